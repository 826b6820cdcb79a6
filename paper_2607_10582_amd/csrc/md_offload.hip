// gfx950 kernels of the offload tier (the second tier of Sec. III-E: pages
// leave the cache for host memory instead of being dropped, and come back
// when later queries make them relevant again).
//
//   k_recall         at an observation, after the attention: every page in
//                    host memory is observed with the step's query, its keys
//                    read straight from the pinned host memory; a token's mass
//                    is its weight 2^(x - M) / Lambda next to the cached tokens
//                    (the rows' normalisers of this step), then EWMA, refresh,
//                    scores (Eq. 2-5); a page with a refreshed token is marked.
//   k_recall_insert  the marked pages come back: a device page each (off the
//                    free list, sessions in order), keys and token state
//                    copied in, merged into the page table in serial order.
//   k_offload        at md_compact: host-memory pages below the drop
//                    threshold are dropped; of the pages the eviction lists,
//                    the full ones at or above it go to host memory, the best
//                    first, while the session's host slots last.
// Sizes: at most kMaxOffload pages per session in host memory (one 64-bit
// mask of host slots).

#include "md_device.h"

namespace md {

namespace {

// The row normalisers (M, 1 / Lambda) of query row `row` of session s at
// this step: the fused kernel's tagged words, or the multi-kernel path's
// row statistics when the session took that path (it then has chunks).
__device__ __forceinline__ float2 row_norm(const Scratch& sc, const Dims& dm, int s, int row, bool fused_norm) {
    if (fused_norm) {
        const unsigned long long* p = sc.unorm + (((size_t)s * dm.R + row) << 1);
        const unsigned long long m = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const unsigned long long inv = __hip_atomic_load(p + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return make_float2(__uint_as_float((uint32_t)m), __uint_as_float((uint32_t)inv));
    }
    return sc.rstats[(size_t)s * dm.R + row];
}

// Unpack eight bf16 values (one 16-byte piece) into floats.
__device__ __forceinline__ void bf16x8_to_f32(const u32x4 x, float* out) {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        out[2 * w] = __uint_as_float(x[w] << 16);
        out[2 * w + 1] = __uint_as_float(x[w] & 0xffff0000u);
    }
}

// Unpack eight FP8 E4M3 codes into floats (exact).
__device__ __forceinline__ void e4m3x8_to_f32(const uint2 x, float* out) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int w = 0; w < 2; ++w) {
        const uint32_t word = w ? x.y : x.x;
        const f32x2 lo = __builtin_amdgcn_cvt_pk_f32_fp8((int)word, false);
        const f32x2 hi = __builtin_amdgcn_cvt_pk_f32_fp8((int)word, true);
        out[4 * w] = lo[0];
        out[4 * w + 1] = lo[1];
        out[4 * w + 2] = hi[0];
        out[4 * w + 3] = hi[1];
    }
}

}  // namespace

// ------------------------------------------------------------ observation

// Grid (H, S), four waves per block: block (i, s) observes the i-th listed
// page of session s.  Wave w takes the (layer, KV head) rows w, w + 4, ...;
// in a row, lane (p, qd) holds token 16 b + p's dims 32 qd .. 32 qd + 31 of
// each 16-token block b and the four quarters add their partial logits with
// shuffles, so every lane of a token ends with the whole logit.
__global__ void __launch_bounds__(256) k_recall(Dims dm, View v, Scratch sc, const float* __restrict__ q) {
    const int s = blockIdx.y, i = blockIdx.x;
    const int H = dm.H;
    if (!sc.valid[s] || i >= min(v.off_count[s], H)) return;
    const int slot = v.off_slot[(size_t)s * H + i];
    if ((unsigned)slot >= (unsigned)H) {
        if (threadIdx.x == 0) atomicOr(sc.status, kDevCorrupt);
        return;
    }
    const unsigned char* page = v.host_keys + ((size_t)s * H + slot) * dm.page_bytes;
    const bool qz = dm.quant && v.off_format[(size_t)s * H + slot];
    const bool fused_norm = sc.chunks[s] == 0;
    const int wv = threadIdx.x >> 6, lane = lane_id();
    const int p = lane & 15, qd = lane >> 4;
    const int nblk = dm.P >> 4;
    __shared__ float part[4][64];
    float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};   // this lane's token of each 16-token block
    // with no cached token the rows have no normalisers: the weights are 0
    const int rows = v.n_live[s] > 0 ? dm.LHkv : 0;
    for (int r = wv; r < rows; r += 4) {
        const int l = r / dm.Hkv, kv = r - l * dm.Hkv;
        for (int b = 0; b < nblk; ++b) {
            const unsigned char* blk = page + ((size_t)r * dm.P + 16 * b) * kHeadDim * 2;
            float k[32];
            float scale = 1.0f;
            if (!qz) {
                // element (t, e) of the block at (e / 8) 128 + t 8 + e % 8
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    bf16x8_to_f32(*reinterpret_cast<const u32x4*>(blk + 2 * ((4 * qd + c) * 128 + p * 8)), k + 8 * c);
            } else {
                // codes of token t, dims 8 c' .. 8 c' + 7 at 1024 (e / 64) +
                // 16 (t + 16 ((e / 8) % 4)) + 8 ((e / 32) % 2); scale at 2048
                scale = *reinterpret_cast<const float*>(blk + 2048);
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    e4m3x8_to_f32(*reinterpret_cast<const uint2*>(blk + 1024 * (qd >> 1) + 16 * (p + 16 * c) + 8 * (qd & 1)),
                                  k + 8 * c);
            }
            for (int h = 0; h < dm.G; ++h) {
                const int row = l * dm.Hq + kv * dm.G + h;
                const f32x4* qh = reinterpret_cast<const f32x4*>(q + ((size_t)s * dm.L * dm.Hq + row) * kHeadDim + 32 * qd);
                float x = 0.0f;
#pragma unroll
                for (int c = 0; c < 8; ++c) {
                    const f32x4 qq = qh[c];
#pragma unroll
                    for (int e = 0; e < 4; ++e) x = fmaf(qq[e], k[4 * c + e], x);
                }
                x += __shfl_xor(x, 16);
                x += __shfl_xor(x, 32);
                x *= scale;
                const float2 nm = row_norm(sc, dm, s, row, fused_norm);
                acc[b] += hw_exp2(x * kLogitScale - nm.x) * nm.y;
            }
        }
    }
    if (qd == 0)
        for (int b = 0; b < nblk; ++b) part[wv][16 * b + p] = acc[b];
    __syncthreads();
    if (wv != 0) return;
    // wave 0, lane t < P: token t of the page
    const int t = lane;
    const bool live = t < dm.P;
    const size_t ts = ((size_t)s * H + slot) * dm.P + (live ? t : 0);
    const int t_now = v.clock[s];
    const int n_tok = v.n_live[s];   // |K_t|: the cached tokens
    float sc_i = 0.0f;
    bool pin = false, refreshed = false;
    if (live) {
        const float abar = (((part[0][t] + part[1][t]) + part[2][t]) + part[3][t]) / (float)dm.R;
        const float a = fmaf(dm.rho, v.off_imp[ts], (1.0f - dm.rho) * abar);
        v.off_imp[ts] = a;
        refreshed = abar >= dm.tau_scale / (float)n_tok;
        int tr;
        if (refreshed) {
            tr = t_now;
            v.off_t_ref[ts] = tr;
        } else {
            tr = v.off_t_ref[ts];
        }
        v.off_abar[ts] = abar;
        int reg = v.off_region[ts];
        if (reg >= dm.n_regions) {
            atomicOr(sc.status, kDevCorrupt);
            reg = dm.n_regions - 1;
        }
        pin = (dm.pin_mask >> reg) & 1u;
        const size_t ri = (size_t)s * dm.n_regions + reg;
        sc_i = pin ? INFINITY
                   : retention_score(v.b[ri], v.lam[ri], t_now, tr, attention_weight(dm.alpha, dm.norm_attn, n_tok), a);
    }
    float ps;
    page_score_of(sc_i, live, pin, dm.P, &ps);
    const bool any = __ballot(refreshed) != 0ull;
    if (lane == 0) {
        v.off_score[(size_t)s * H + i] = ps;
        sc.recall[(size_t)s * H + i] = any ? 1 : 0;
        if (any) atomicAdd(sc.rcount + s, 1);
        atomicAdd(&sc.counters[7], 1ull);
    }
}

// Copy `bytes` (a multiple of 16) from src to dst with the whole block.
__device__ __forceinline__ void block_copy(unsigned char* __restrict__ dst, const unsigned char* __restrict__ src,
                                           size_t bytes) {
    const size_t n = bytes >> 4;
    for (size_t j = threadIdx.x; j < n; j += blockDim.x)
        reinterpret_cast<u32x4*>(dst)[j] = reinterpret_cast<const u32x4*>(src)[j];
}

// Pages session s2 can take back at this step: its marked pages, as far as
// its page table has room (counts as they stand before any recall).
__device__ __forceinline__ int recall_room(const Dims& dm, const View& v, const Scratch& sc, int s2) {
    return min(sc.rcount[s2], max(dm.MP - v.n_pages[s2], 0));
}

// One block per session: the pages k_recall marked come back, as many as
// the page table has room for (the first in serial order).  Pages leave the
// free list in session order, after those of the sessions before (their
// recall counts are final: k_recall ran in an earlier launch, and no block
// changes a page count before the last block).  The page table, the serials
// and the library's page scores are merged in serial order; the recalled
// pages are full, and their serials lie below the last page's, so only the
// last page stays partial.
__global__ void __launch_bounds__(kSelThreads) k_recall_insert(Dims dm, View v, Scratch sc, float* abar_out) {
    const int s = blockIdx.x;
    const int H = dm.H;
    const int tid = threadIdx.x;
    __shared__ int sh_before, sh_last, sh_r;
    __shared__ int r_serial[kMaxOffload], r_phys[kMaxOffload], r_slot[kMaxOffload], r_pos[kMaxOffload];
    __shared__ float r_score[kMaxOffload];
    __shared__ int lds[17];
    if (tid == 0) {
        sh_before = 0;
        sh_r = 0;
    }
    __syncthreads();
    {
        int mine = 0;
        for (int s2 = tid; s2 < s; s2 += blockDim.x) mine += recall_room(dm, v, sc, s2);
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) mine += __shfl_xor(mine, o);
        if (lane_id() == 0 && mine > 0) atomicAdd(&sh_before, mine);
    }
    __syncthreads();
    const int room_s = recall_room(dm, v, sc, s);
    const bool ok = sc.valid[s] && room_s > 0;
    const int cnt = min(v.off_count[s], H);
    const int fc = v.free_count[0];   // changes only in the last block
    // wave 0: the recalled entries in list (serial) order, their pops
    if (ok && tid < 64) {
        const bool marked = tid < cnt && sc.recall[(size_t)s * H + tid] != 0;
        const unsigned long long mm = __ballot(marked);
        const bool flag = marked && __popcll(mm & ((1ull << tid) - 1ull)) < room_s;
        const unsigned long long m = __ballot(flag);
        const int k = __popcll(m & ((1ull << tid) - 1ull));
        if (flag) {
            const int idx = min(fc, dm.NP) - 1 - (sh_before + k);
            const int phys = idx >= 0 ? v.free_list[idx] : -1;
            r_serial[k] = v.off_serial[(size_t)s * H + tid];
            r_slot[k] = v.off_slot[(size_t)s * H + tid];
            r_score[k] = v.off_score[(size_t)s * H + tid];
            r_phys[k] = (phys >= 0 && phys < dm.NP) ? phys : -1;
            r_pos[k] = tid;
            if (idx < 0) atomicOr(sc.status, MD_DEV_CAPACITY);
            else if (phys < 0 || phys >= dm.NP) atomicOr(sc.status, kDevCorrupt);
        }
        if (tid == 0) sh_r = __popcll(m);
    }
    __syncthreads();
    const int r_all = sh_r;
    // pages that found no device page stay in host memory; the rest
    // (a prefix of the recalled entries: pops go down the stack in order)
    int r = 0;
    while (r < r_all && r_phys[r] >= 0) ++r;
    for (int k = 0; k < r; ++k) {
        const int phys = r_phys[k];
        const int slot = r_slot[k];
        block_copy(reinterpret_cast<unsigned char*>(v.k_pool) + (size_t)phys * dm.page_bytes,
                   v.host_keys + ((size_t)s * H + slot) * dm.page_bytes, dm.page_bytes);
        if (tid < dm.P) {
            const size_t src = ((size_t)s * H + slot) * dm.P + tid;
            const size_t dst = (size_t)phys * dm.P + tid;
            v.region[dst] = v.off_region[src];
            v.t_ins[dst] = v.off_t_ins[src];
            v.t_ref[dst] = v.off_t_ref[src];
            v.imp[dst] = v.off_imp[src];
            if (abar_out != nullptr) abar_out[dst] = v.off_abar[src];
        }
        if (tid == 0 && dm.quant) v.page_format[phys] = v.off_format[(size_t)s * H + slot];
    }
    // merge into the page table (every read before any write)
    const int np0 = v.n_pages[s];
    const int np = ok ? np0 : 0;
    const int per = (np + kSelThreads - 1) / kSelThreads;
    const int i0 = min(np, tid * per), i1 = min(np, i0 + per);
    int32_t* ptab = v.page_table + (size_t)s * dm.MP;
    int32_t* pser = v.page_serial + (size_t)s * dm.MP;
    float* psc = sc.pscore + (size_t)s * dm.MP;
    int ph[kPerThread], se[kPerThread];
    float pv[kPerThread];
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) {
        ph[k] = se[k] = 0;
        pv[k] = 0.0f;
        if (i0 + k < i1) {
            ph[k] = ptab[i0 + k];
            se[k] = pser[i0 + k];
            pv[k] = psc[i0 + k];
        }
    }
    int rp = 0;   // recalled entry k's new index (threads k < r)
    if (tid < r) {
        int lo = 0, hi = np;   // cached pages with a smaller serial
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (pser[mid] < r_serial[tid]) lo = mid + 1; else hi = mid;
        }
        rp = tid + lo;
    }
    // the host-memory list without the recalled entries (wave 0)
    int keep_ser = 0, keep_slot = 0, keep_pos = -1;
    float keep_score = 0.0f;
    if (ok && r > 0 && tid < 64) {
        bool gone = false;
        for (int k = 0; k < r; ++k) gone |= r_pos[k] == tid;
        const bool keep = tid < cnt && !gone;
        const unsigned long long m = __ballot(keep);
        if (keep) {
            keep_pos = __popcll(m & ((1ull << tid) - 1ull));
            keep_ser = v.off_serial[(size_t)s * H + tid];
            keep_slot = v.off_slot[(size_t)s * H + tid];
            keep_score = v.off_score[(size_t)s * H + tid];
        }
    }
    __syncthreads();
    if (ok && r > 0) {
#pragma unroll
        for (int k = 0; k < kPerThread; ++k) {
            if (i0 + k < i1) {
                int before = 0;   // recalled pages with a smaller serial
                for (int j = 0; j < r; ++j) before += r_serial[j] < se[k] ? 1 : 0;
                const int ni = i0 + k + before;
                ptab[ni] = ph[k];
                pser[ni] = se[k];
                psc[ni] = pv[k];
            }
        }
        if (tid < r) {
            ptab[rp] = r_phys[tid];
            pser[rp] = r_serial[tid];
            psc[rp] = r_score[tid];
        }
        if (keep_pos >= 0) {
            v.off_serial[(size_t)s * H + keep_pos] = keep_ser;
            v.off_slot[(size_t)s * H + keep_pos] = keep_slot;
            v.off_score[(size_t)s * H + keep_pos] = keep_score;
        }
        if (tid == 0) {
            v.off_count[s] = cnt - r;
            atomicAdd(sc.opened, r);
            atomicAdd(&sc.counters[5], (unsigned long long)r);
        }
    }
    // the new page count, applied by the last block (the ranks above read
    // the counts before any recall)
    if (tid == 0) sc.freed[s] = (ok && r > 0) ? r : 0;
    // The last block: the pages taken off the free list, and the recall
    // counts cleared for the next observation.
    __threadfence();
    __syncthreads();
    if (tid == 0) sh_last = (atomicAdd(sc.done_compact, 1) == (int)gridDim.x - 1);
    __syncthreads();
    if (!sh_last) return;
    __threadfence();
    if (tid == 0) {
        const int taken = load_agent(sc.opened);
        v.free_count[0] = max(min(fc, dm.NP) - taken, 0);
        *sc.opened = 0;
        *sc.done_compact = 0;
    }
    // new page and token counts, and the scoring kernel's work list (its
    // 64-token tiles per session, laid out by the append) grown to match
    int tiles = 0;
    if (tid < dm.S) {
        const int back = load_agent(sc.freed + tid);
        tiles = sc.score_prefix[tid + 1] - sc.score_prefix[tid];
        if (back > 0) {
            const int nt_old = v.n_tokens[tid];
            const int nt_new = nt_old + back * dm.P;
            v.n_pages[tid] += back;
            v.n_tokens[tid] = nt_new;
            tiles += (nt_new + kTile - 1) / kTile - (nt_old + kTile - 1) / kTile;
        }
        sc.rcount[tid] = 0;
    }
    int total;
    const int ex = block_exclusive_scan(tiles, lds, &total);
    if (tid < dm.S) sc.score_prefix[tid] = ex;
    if (tid == 0) sc.score_prefix[dm.S] = total;
}

hipError_t launch_recall(const Dims& dm, const View& v, const Scratch& sc, const float* q, float* abar_out,
                         hipStream_t st) {
    hipLaunchKernelGGL(k_recall, dim3(dm.H, dm.S), dim3(256), 0, st, dm, v, sc, q);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_recall_insert, dim3(dm.S), dim3(kSelThreads), 0, st, dm, v, sc, abar_out);
    return hipGetLastError();
}

// ------------------------------------------------------------ offload

// One block per session, at md_compact before the quantised tier and the
// compaction (the device pages are freed by the compaction, after their keys
// were copied out here).
//  1. host-memory pages scoring below the drop threshold are dropped;
//  2. candidates: pages on the eviction list that take no more tokens (all
//     but the last page, or a full last page) and score at least the
//     threshold;
//  3. the best `room` of them (room = free host slots) by a radix select
//     over the complemented float bits (descending scores), pages with the
//     threshold key in page order, i.e. the older first;
//  4. their keys go to the lowest free host slots in serial order, their
//     tokens' state with them, and the list is merged in serial order.
__global__ void __launch_bounds__(kSelThreads) k_offload(Dims dm, View v, Scratch sc,
                                                         const int32_t* __restrict__ ev_serial,
                                                         const int32_t* __restrict__ ev_count) {
    const int s = blockIdx.x;
    const int H = dm.H;
    const int tid = threadIdx.x;
    __shared__ int lds[17];
    __shared__ int hist[256];
    __shared__ int sh_digit, sh_before, sh_kept, sh_nc;
    __shared__ unsigned long long sh_used;
    __shared__ int c_idx[kMaxOffload], c_slot[kMaxOffload], c_ser[kMaxOffload], kept_ser[kMaxOffload];
    if (!sc.valid[s]) return;
    const int cnt_off = min(v.off_count[s], H);
    // 1. drops: wave 0 holds the list; the kept entries stay in registers
    // until the merge
    int k_ser = 0, k_slot = 0, k_pos = -1;
    float k_score = 0.0f;
    if (tid < 64) {
        const bool in = tid < cnt_off;
        const float sc0 = in ? v.off_score[(size_t)s * H + tid] : 0.0f;
        const bool keep = in && sc0 >= dm.drop_thr;
        const unsigned long long m = __ballot(keep);
        unsigned long long used = 0ull;
        if (keep) {
            k_pos = __popcll(m & ((1ull << tid) - 1ull));
            k_ser = v.off_serial[(size_t)s * H + tid];
            k_slot = v.off_slot[(size_t)s * H + tid];
            k_score = sc0;
            kept_ser[k_pos] = k_ser;
            used = 1ull << (k_slot & 63);
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) used |= __shfl_xor(used, o);
        if (tid == 0) {
            sh_kept = __popcll(m);
            sh_used = used;
            atomicAdd(&sc.counters[6], (unsigned long long)(cnt_off - __popcll(m)));
        }
    }
    __syncthreads();
    const int kept = sh_kept;
    const int room = H - kept;
    // 2. candidates
    const int np = v.n_pages[s], nt = v.n_tokens[s];
    const int cnt = min(max(ev_count[s], 0), dm.MP);
    const int32_t* evs = ev_serial + (size_t)s * dm.MP;
    const int32_t* ptab = v.page_table + (size_t)s * dm.MP;
    const int32_t* pser = v.page_serial + (size_t)s * dm.MP;
    const float* psc = sc.pscore + (size_t)s * dm.MP;
    const int per = (np + kSelThreads - 1) / kSelThreads;
    const int i0 = min(np, tid * per), i1 = min(np, i0 + per);
    uint32_t key[kPerThread];
    bool cand[kPerThread];
    int ncand = 0;
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) {
        const int i = i0 + k;
        key[k] = 0u;
        cand[k] = false;
        if (i < i1 && cnt > 0 && room > 0) {
            int lo = 0, hi = cnt;
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (evs[mid] < pser[i]) lo = mid + 1; else hi = mid;
            }
            const bool gone = lo < cnt && evs[lo] == pser[i];
            const bool full = i < np - 1 || nt == np * dm.P;
            const float v0 = psc[i];
            if (gone && full && v0 >= dm.drop_thr && v0 < INFINITY) {
                key[k] = ~__float_as_uint(v0);   // non-negative scores: descending order
                cand[k] = true;
                ++ncand;
            }
        }
    }
    int total;
    block_exclusive_scan(ncand, lds, &total);
    const int need = min(total, max(room, 0));
    // 3. radix select of the `need` smallest keys (threshold key T; the
    // pages with key T in page order)
    uint32_t T = 0xFFFFFFFFu;
    int rem = need;
    if (need > 0 && need < total) {
        uint32_t prefix = 0, pmask = 0;
        for (int shift = 24; shift >= 0; shift -= 8) {
            if (tid < 256) hist[tid] = 0;
            __syncthreads();
#pragma unroll
            for (int k = 0; k < kPerThread; ++k)
                if (cand[k] && (key[k] & pmask) == prefix) atomicAdd(&hist[(key[k] >> shift) & 255u], 1);
            __syncthreads();
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
    }
    int teq = 0;
#pragma unroll
    for (int k = 0; k < kPerThread; ++k)
        if (cand[k] && need < total && key[k] == T) ++teq;
    int dummy;
    int run = block_exclusive_scan(teq, lds, &dummy);
    bool pick[kPerThread];
    int my_pick = 0;
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) {
        bool e = false;
        if (cand[k] && need > 0) {
            if (need >= total || key[k] < T) {
                e = true;
            } else if (key[k] == T) {
                e = run < rem;
                ++run;
            }
        }
        pick[k] = e;
        my_pick += e ? 1 : 0;
    }
    int n_pick;
    int pos = block_exclusive_scan(my_pick, lds, &n_pick);
    // the chosen pages in serial (page) order and their host slots: the
    // lowest free slots in turn
#pragma unroll
    for (int k = 0; k < kPerThread; ++k)
        if (pick[k] && pos < kMaxOffload) c_idx[pos++] = i0 + k;
    if (tid == 0) sh_nc = min(n_pick, kMaxOffload);
    __syncthreads();
    const int nc = sh_nc;
    if (tid < 64) {
        const unsigned long long all = H >= 64 ? ~0ull : ((1ull << H) - 1ull);
        unsigned long long freem = all & ~sh_used;
        // the tid-th set bit of freem
        int slot = -1;
        for (int j = 0; j <= tid && freem != 0ull; ++j) {
            const int b = __ffsll((long long)freem) - 1;
            if (j == tid) slot = b;
            freem &= freem - 1ull;
        }
        if (tid < nc) c_slot[tid] = slot;
    }
    __syncthreads();
    // 4. copy out, token state, list merge
    for (int k = 0; k < nc; ++k) {
        const int i = c_idx[k];
        const int phys = ptab[i];
        const int slot = c_slot[k];
        if ((unsigned)phys >= (unsigned)dm.NP || slot < 0) {
            if (tid == 0) atomicOr(sc.status, kDevCorrupt);
            continue;
        }
        block_copy(v.host_keys + ((size_t)s * H + slot) * dm.page_bytes,
                   reinterpret_cast<const unsigned char*>(v.k_pool) + (size_t)phys * dm.page_bytes, dm.page_bytes);
        if (tid < dm.P) {
            const size_t src = (size_t)phys * dm.P + tid;
            const size_t dst = ((size_t)s * H + slot) * dm.P + tid;
            v.off_region[dst] = v.region[src];
            v.off_t_ins[dst] = v.t_ins[src];
            v.off_t_ref[dst] = v.t_ref[src];
            v.off_imp[dst] = v.imp[src];
            v.off_abar[dst] = 0.0f;
        }
        if (tid == 0) v.off_format[(size_t)s * H + slot] = dm.quant ? v.page_format[phys] : 0;
    }
    // merge: kept entries (wave 0, registers) and chosen pages, by serial
    if (tid < nc) c_ser[tid] = pser[c_idx[tid]];
    __syncthreads();
    if (k_pos >= 0) {
        int before = 0;   // chosen pages with a smaller serial
        for (int k = 0; k < nc; ++k) before += c_ser[k] < k_ser ? 1 : 0;
        const size_t ni = (size_t)s * H + k_pos + before;
        v.off_serial[ni] = k_ser;
        v.off_slot[ni] = k_slot;
        v.off_score[ni] = k_score;
    }
    if (tid < nc) {
        int before = 0;   // kept entries with a smaller serial
        for (int j = 0; j < kept; ++j) before += kept_ser[j] < c_ser[tid] ? 1 : 0;
        const size_t ni = (size_t)s * H + tid + before;
        v.off_serial[ni] = c_ser[tid];
        v.off_slot[ni] = c_slot[tid];
        v.off_score[ni] = psc[c_idx[tid]];
    }
    if (tid == 0) {
        v.off_count[s] = kept + nc;
        atomicAdd(&sc.counters[4], (unsigned long long)nc);
    }
}

hipError_t launch_offload(const Dims& dm, const View& v, const Scratch& sc, const int32_t* ev_serial,
                          const int32_t* ev_count, hipStream_t st) {
    hipLaunchKernelGGL(k_offload, dim3(dm.S), dim3(kSelThreads), 0, st, dm, v, sc, ev_serial, ev_count);
    return hipGetLastError();
}

}  // namespace md
