// C-ABI layer of the MemDecay retention step: argument validation (all on the
// host, before anything is enqueued), the handle, the scratch, and the order
// of kernel launches on the caller's stream.

#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <new>
#include <vector>

#include "md_internal.h"

namespace {

enum Phase { kNone = 0, kObserved = 1, kScored = 2, kCompacted = 3 };

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace

struct Timed {
    hipEvent_t start, stop;
};

struct md_handle_s {
    md::Dims dm;
    md::View v;
    md::Scratch sc;
    hipStream_t stream;
    int device;
    void* scratch;
    int logits_blocks;
    int mass_blocks;
    int score_blocks;
    bool have_step;
    int32_t last_step;
    bool fused_first;    // the first observe runs the fused kernel
    bool fused_steady;   // later observes run the fused kernel
    int rg_first;        // row groups of the fused units on the first observe
    int rg_steady;       // and on later ones (1: every unit walks every row)
    int64_t observed;    // observes enqueued
    Phase phase;
    const int32_t* sel_serial;   // md_select_evict's lists since the last observe
    const int32_t* sel_count;    // (NULL: no selection yet)
    uint32_t profile_mask;
    std::vector<Timed> pending[MD_K_COUNT];   // launches not yet read back
    std::vector<Timed> spare;                  // recycled event pairs
    int static_slot;     // md_init_static: index in the static handles; -1 otherwise
    uint32_t word_tag; // tag of the last launch handing counts between blocks through tagged words
};

namespace {

// Handles of md_init_static live here, so that it allocates no host memory
// either; a slot is taken by md_init_static and given back by md_destroy.
constexpr int kStaticHandles = 16;
md_handle_s g_static_handles[kStaticHandles];
std::atomic<bool> g_static_taken[kStaticHandles];

md_handle_s* take_static_handle() {
    for (int i = 0; i < kStaticHandles; ++i) {
        bool expect = false;
        if (g_static_taken[i].compare_exchange_strong(expect, true)) {
            md_handle_s* h = &g_static_handles[i];
            h->static_slot = i;
            return h;
        }
    }
    return nullptr;
}

void give_back(md_handle_s* h) {
    if (h->static_slot < 0) {
        delete h;
        return;
    }
    const int i = h->static_slot;
    for (auto& v : h->pending) v.clear();
    h->spare.clear();
    h->profile_mask = 0;
    g_static_taken[i].store(false);
}

// Launch through `fn(start, stop)`, timed by an event pair when kernel `id`
// is timed.  With `inside` the launch records the pair itself
// (hipExtLaunchKernel: the events take the kernel's own start and end, with
// no packets of their own in the stream); otherwise fn gets (NULL, NULL)
// and the pair is recorded around it.
template <typename F>
hipError_t timed_launch_ev(md_handle_s* h, int id, bool inside, F&& fn) {
    if (!(h->profile_mask & (1u << id))) return fn(nullptr, nullptr);
    Timed t;
    if (!h->spare.empty()) {
        t = h->spare.back();
        h->spare.pop_back();
    } else {
        // timing only: no system-scope fence (cache writeback and
        // invalidation) when the event is recorded, which would slow the
        // work after it and inflate the figure
        if (hipEventCreateWithFlags(&t.start, hipEventDisableSystemFence) != hipSuccess) return hipErrorOutOfMemory;
        if (hipEventCreateWithFlags(&t.stop, hipEventDisableSystemFence) != hipSuccess) {
            (void)hipEventDestroy(t.start);
            return hipErrorOutOfMemory;
        }
    }
    hipError_t e;
    if (inside) {
        e = fn(t.start, t.stop);
    } else {
        e = hipEventRecord(t.start, h->stream);
        if (e == hipSuccess) e = fn(nullptr, nullptr);
        if (e == hipSuccess) e = hipEventRecord(t.stop, h->stream);
    }
    if (e == hipSuccess) h->pending[id].push_back(t); else h->spare.push_back(t);
    return e;
}

template <typename F>
hipError_t timed_launch(md_handle_s* h, int id, F&& fn) {
    return timed_launch_ev(h, id, false, [&](hipEvent_t, hipEvent_t) { return fn(); });
}

// Tag of the next launch that hands counts between its blocks through
// tagged words (the append, the one-launch select-and-compact): never 0 (the
// scratch starts zeroed) and never the previous one.
uint32_t next_word_tag(md_handle_s* h) {
    h->word_tag = (h->word_tag % md::kWordTagMask) + 1;
    return h->word_tag;
}

void release_events(md_handle_s* h) {
    for (auto& v : h->pending) {
        for (auto& t : v) h->spare.push_back(t);
        v.clear();
    }
    for (auto& t : h->spare) {
        (void)hipEventDestroy(t.start);
        (void)hipEventDestroy(t.stop);
    }
    h->spare.clear();
}

}  // namespace

extern "C" {

int32_t md_abi_version(void) { return MD_ABI_VERSION; }

const char* md_status_str(md_status s) {
    switch (s) {
        case MD_OK: return "ok";
        case MD_E_INVALID: return "invalid argument (null or misaligned pointer, or a value out of range)";
        case MD_E_UNSUPPORTED: return "unsupported shape (head_dim must be 128, page_size 16 or 64, "
                                      "Hq/Hkv <= 16, L*Hq <= 1024, sessions <= 1024, pages per session <= 8192)";
        case MD_E_STEP: return "step must advance by exactly one per md_observe_step";
        case MD_E_HIP: return "HIP runtime call failed";
        case MD_E_STATE: return "call out of order (score needs an observe, select needs a score, "
                                "and neither may follow a compact before the next observe)";
        case MD_E_NOMEM: return "could not allocate the library scratch";
        case MD_E_TOO_LARGE: return "the handle's scratch exceeds md_init_static's static scratch (128 MiB), "
                                    "or all 16 static handles are in use";
        case MD_W_BUDGET_INFEASIBLE: return "warning: a session's pinned tokens exceed its budget";
        default: return "unknown status";
    }
}

static md_status validate_config(const md_config* c) {
    if (c == nullptr) return MD_E_INVALID;
    if ((c->flags & ~(MD_FLAG_NO_FUSED | MD_FLAG_FUSED | MD_FLAG_NORM_ATTENTION | MD_FLAG_REGION_ALIGNED |
                      MD_FLAG_COOPERATIVE | MD_FLAG_NO_ROW_GROUPS)) != 0)
        return MD_E_INVALID;
    if ((c->flags & MD_FLAG_NO_FUSED) && (c->flags & MD_FLAG_FUSED)) return MD_E_INVALID;
    if (c->offload_pages < 0 || c->offload_pages > md::kMaxOffload) return MD_E_INVALID;
    if (!(c->drop_threshold >= 0.0f)) return MD_E_INVALID;   // NaN too
    // the offload tier runs with one query per observation on plain pages
    if (c->offload_pages > 0 && (c->window > 1 || (c->flags & MD_FLAG_REGION_ALIGNED))) return MD_E_UNSUPPORTED;
    if (c->n_layers < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1) return MD_E_INVALID;
    if (c->n_q_heads % c->n_kv_heads != 0) return MD_E_INVALID;
    if (c->max_sessions < 1 || c->max_pages < 1 || c->n_phys_pages < 1) return MD_E_INVALID;
    if (c->n_regions < 1 || c->n_regions > 32) return MD_E_INVALID;
    if (c->n_regions < 32 && (c->pinned_region_mask >> c->n_regions) != 0) return MD_E_INVALID;
    if (!(c->rho >= 0.0f && c->rho < 1.0f)) return MD_E_INVALID;
    if (!(c->alpha >= 0.0f) || !isfinite(c->alpha)) return MD_E_INVALID;
    if (!(c->tau_scale >= 0.0f) || !isfinite(c->tau_scale)) return MD_E_INVALID;
    if (c->window < 1) return MD_E_INVALID;
    if (!(c->quant_threshold >= 0.0f)) return MD_E_INVALID;   // NaN too
    if (c->head_dim != md::kHeadDim) return MD_E_UNSUPPORTED;
    if ((int64_t)(c->n_q_heads / c->n_kv_heads) * c->window > 16) return MD_E_UNSUPPORTED;
    if ((int64_t)c->n_layers * c->n_q_heads * c->window > md::kMaxRows) return MD_E_UNSUPPORTED;
    if (c->page_size != 16 && c->page_size != 64) return MD_E_UNSUPPORTED;
    if (c->n_q_heads / c->n_kv_heads > 16) return MD_E_UNSUPPORTED;
    if ((int64_t)c->n_layers * c->n_q_heads > md::kMaxRows) return MD_E_UNSUPPORTED;
    if (c->max_sessions > md::kMaxSessions) return MD_E_UNSUPPORTED;
    if (c->max_pages > md::kMaxPages) return MD_E_UNSUPPORTED;
    // token and element counts must stay within int32 where kernels index with int
    if ((int64_t)c->max_pages * c->page_size > (int64_t)1 << 30) return MD_E_UNSUPPORTED;
    if ((int64_t)c->n_phys_pages * c->page_size > (int64_t)1 << 30) return MD_E_UNSUPPORTED;
    return MD_OK;
}

static md_status validate_view(const md_cache_view* v, bool region_aligned, bool quant, bool offload) {
    if (v == nullptr) return MD_E_INVALID;
    if (quant && v->page_format == nullptr) return MD_E_INVALID;
    if (offload) {
        const void* op[] = {v->host_keys, v->off_count, v->off_serial, v->off_slot, v->off_region, v->off_t_ins,
                            v->off_t_ref, v->off_importance, v->off_format, v->off_score, v->off_abar};
        for (const void* p : op)
            if (p == nullptr) return MD_E_INVALID;
        const void* ow[] = {v->host_keys, v->off_count, v->off_serial, v->off_slot, v->off_t_ins, v->off_t_ref,
                            v->off_importance, v->off_score, v->off_abar};
        for (const void* p : ow)
            if (!aligned(p, 16 / (p == v->host_keys ? 1 : 4))) return MD_E_INVALID;
    }
    if (region_aligned && (v->n_live == nullptr || !aligned(v->n_live, 4) || !aligned(v->region, 4)))
        return MD_E_INVALID;
    const void* ptrs[] = {v->k_pool, v->region, v->t_ins, v->t_ref, v->importance,
                          v->page_table, v->page_serial, v->n_pages, v->n_tokens, v->clock,
                          v->next_serial, v->budget, v->free_list, v->free_count};
    for (const void* p : ptrs)
        if (p == nullptr) return MD_E_INVALID;
    if (!aligned(v->k_pool, 16)) return MD_E_INVALID;
    const void* words[] = {v->t_ins, v->t_ref, v->importance, v->page_table, v->page_serial,
                           v->n_pages, v->n_tokens, v->clock, v->next_serial, v->budget,
                           v->free_list, v->free_count};
    for (const void* p : words)
        if (!aligned(p, 4)) return MD_E_INVALID;
    return MD_OK;
}

// md_init and md_init_static: use_static takes the scratch from the
// library's static device array and the handle from the static handles.
static md_status init_handle(const md_config* cfg, const md_region_params* rp, const md_cache_view* cv,
                             void* stream, md_handle* out, bool use_static) {
    if (out == nullptr) return MD_E_INVALID;
    *out = nullptr;
    md_status st = validate_config(cfg);
    if (st != MD_OK) return st;
    st = validate_view(cv, (cfg->flags & MD_FLAG_REGION_ALIGNED) != 0, cfg->quant_threshold > 0.0f,
                       cfg->offload_pages > 0);
    if (st != MD_OK) return st;
    if (rp == nullptr || rp->base_priority == nullptr || rp->decay_rate == nullptr) return MD_E_INVALID;
    if (!aligned(rp->base_priority, 4) || !aligned(rp->decay_rate, 4)) return MD_E_INVALID;

    md::Dims dm{};
    dm.L = cfg->n_layers;
    dm.Hq = cfg->n_q_heads;
    dm.Hkv = cfg->n_kv_heads;
    dm.G = dm.Hq / dm.Hkv;
    dm.P = cfg->page_size;
    dm.Pshift = dm.P == 16 ? 4 : 6;
    dm.S = cfg->max_sessions;
    dm.MP = cfg->max_pages;
    dm.NP = cfg->n_phys_pages;
    dm.W = cfg->window;
    dm.R = dm.L * dm.Hq * dm.W;   // softmax rows: (layer, query head, window query)
    dm.LHkv = dm.L * dm.Hkv;
    dm.n_regions = cfg->n_regions;
    dm.max_chunks = (int)(((int64_t)dm.MP * dm.P + md::kChunk - 1) / md::kChunk);
    dm.pin_mask = cfg->pinned_region_mask;
    dm.rho = cfg->rho;
    dm.alpha = cfg->alpha;
    dm.tau_scale = cfg->tau_scale;
    dm.fused = (cfg->flags & MD_FLAG_NO_FUSED) ? 0 : 1;
    dm.norm_attn = (cfg->flags & MD_FLAG_NORM_ATTENTION) ? 1 : 0;
    dm.coop = (cfg->flags & MD_FLAG_COOPERATIVE) ? 1 : 0;
    dm.aligned = (cfg->flags & MD_FLAG_REGION_ALIGNED) ? 1 : 0;
    dm.quant = cfg->quant_threshold > 0.0f ? 1 : 0;
    dm.quant_thr = cfg->quant_threshold;
    dm.H = cfg->offload_pages;
    dm.drop_thr = cfg->drop_threshold;
    dm.page_bytes = (size_t)dm.LHkv * dm.P * md::kHeadDim * sizeof(uint16_t);

    // ---- from here on the HIP runtime is used
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return MD_E_HIP;
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return MD_E_HIP;
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) return MD_E_UNSUPPORTED;
    hipStream_t hs = static_cast<hipStream_t>(stream);

    // Region priors: b_r >= 0, lambda_r >= 0, finite (Sec. III-B); read in
    // chunks through buffers on the stack.
    const size_t nrp = (size_t)dm.S * dm.n_regions;
    {
        constexpr size_t kChunkN = 2048;
        float hb[kChunkN], hl[kChunkN];
        for (size_t o = 0; o < nrp; o += kChunkN) {
            const size_t n = std::min(kChunkN, nrp - o);
            if (hipMemcpyAsync(hb, rp->base_priority + o, n * sizeof(float), hipMemcpyDeviceToHost, hs) !=
                    hipSuccess ||
                hipMemcpyAsync(hl, rp->decay_rate + o, n * sizeof(float), hipMemcpyDeviceToHost, hs) != hipSuccess ||
                hipStreamSynchronize(hs) != hipSuccess)
                return MD_E_HIP;
            for (size_t i = 0; i < n; ++i)
                if (!(hb[i] >= 0.0f) || !isfinite(hb[i]) || !(hl[i] >= 0.0f) || !isfinite(hl[i]))
                    return MD_E_INVALID;
        }
    }
    void* static_base = nullptr;
    if (use_static && md::static_scratch(&static_base) != hipSuccess) return MD_E_HIP;

    // Fused observation kernel: up to kAttendPerCu workgroups per CU, as
    // many as its LDS and registers allow; md_init then checks on the device
    // that all of them are resident at once.
    const int n_cu = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 256;
    int occ = 0;
    dm.T = md::attend_unit_tokens(dm.G);
    // Row groups (plain pages, one query per observation): their own
    // instantiation, used only if it is as resident as the plain one.
    bool rows_ok = dm.fused && !dm.aligned && !dm.quant && dm.W == 1 && !(cfg->flags & MD_FLAG_NO_ROW_GROUPS) &&
                   dm.LHkv >= 2 * md::kMinGroupRows;
    if (dm.fused) {
        const size_t lds = md::attend_lds_bytes(dm.G * dm.W);
        auto occupancy = [&](int rg, int* o) {
            const void* fn = md::attend_kernel(dm.G * dm.W, dm.aligned, dm.quant, dm.W, rg);
            *o = 0;
            if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess) {
                (void)hipGetLastError();
                return hipSuccess;
            }
            return hipOccupancyMaxActiveBlocksPerMultiprocessor(o, fn, md::attend_threads(dm.G * dm.W), lds);
        };
        if (occupancy(1, &occ) != hipSuccess) return MD_E_HIP;
        if (occ > md::kAttendPerCu) occ = md::kAttendPerCu;
        if (rows_ok) {
            int occ_rg = 0;
            if (occupancy(2, &occ_rg) != hipSuccess) return MD_E_HIP;
            rows_ok = occ_rg >= occ;
        }
        dm.n_wg = occ * n_cu;
        dm.fused = occ >= 1;
    }
    if (dm.fused) {
        dm.U_cap = (int)(((int64_t)dm.NP * dm.P + dm.T - 1) / dm.T + dm.S);
    } else {
        dm.n_wg = dm.U_cap = dm.wg_per_cu = dm.lane_cap = 0;
    }
    // The fused kernel's workgroups wait for each other, so all of them must
    // be resident together: check it on the device, with the launch kind the
    // step uses, and step the grid down one workgroup per CU at a time until
    // every workgroup arrives.
    int32_t* probe = nullptr;   // kept for the row-group instantiation's check below
    auto free_probe = [&] {
        if (!use_static && probe != nullptr) (void)hipFree(probe);
        probe = nullptr;
    };
    if (dm.fused) {
        probe = static_cast<int32_t*>(static_base);   // the static scratch is free until carved
        if (!use_static && hipMalloc(&probe, 2 * sizeof(int32_t)) != hipSuccess) return MD_E_NOMEM;
        int verified = 0;
        for (int o = occ; o >= 1 && verified == 0; --o) {
            int32_t seen[2] = {0, 0};
            if (md::launch_attend_check(dm, probe, o * n_cu, 1, hs) != hipSuccess ||
                hipMemcpyAsync(seen, probe, sizeof(seen), hipMemcpyDeviceToHost, hs) != hipSuccess ||
                hipStreamSynchronize(hs) != hipSuccess) {
                (void)hipGetLastError();
                continue;
            }
            if (seen[1] >= o * n_cu) verified = o * n_cu;
        }
        dm.n_wg = verified;
        dm.wg_per_cu = verified / n_cu;
        dm.lane_cap = n_cu;
        dm.fused = verified > 0;
        if (!dm.fused) dm.U_cap = 0;
    }
    dm.spill = !dm.fused || (int64_t)dm.MP * dm.P > (int64_t)dm.n_wg * dm.T;

    // Path of the first observe and of the later ones.  The fused kernel walks
    // the L * Hkv key rows of each unit in order, a few microseconds per row,
    // so it pays off once its units fill half its workgroups; below that the
    // multi-kernel path, parallel over rows, is faster.  Units are counted
    // from the cache's sizes now (first observe) and with each session at
    // most one token over its budget (later observes, once evictions hold
    // the budget).
    // Row groups: when a step's units fill less than half of the grid, each
    // unit covers one of rg ranges of at least kMinGroupRows rows, rg as
    // large as the grid takes (sessions of the page table's capacity still
    // fit one pass); the fused kernel then runs for steps whose units, times
    // rg, fill a quarter of the grid.
    bool fused_first = dm.fused, fused_steady = dm.fused;
    int rg_first = 1, rg_steady = 1;
    if (dm.fused) {
        int32_t hn[md::kMaxSessions], hbud[md::kMaxSessions];
        if (hipMemcpyAsync(hn, cv->n_tokens, dm.S * sizeof(int32_t), hipMemcpyDeviceToHost, hs) != hipSuccess ||
            hipMemcpyAsync(hbud, cv->budget, dm.S * sizeof(int32_t), hipMemcpyDeviceToHost, hs) !=
                hipSuccess ||
            hipStreamSynchronize(hs) != hipSuccess) {
            free_probe();
            return MD_E_HIP;
        }
        int64_t first = 0, steady = 0;
        for (int s = 0; s < dm.S; ++s) {
            const int64_t n = hn[s] > 0 ? hn[s] : 0;
            const int64_t b = hbud[s] >= 0 ? (int64_t)hbud[s] + 1 : n;
            first += (n + dm.T - 1) / dm.T;
            steady += (std::min(n, b) + dm.T - 1) / dm.T;
        }
        const int64_t cap_units = ((int64_t)dm.MP * dm.P + dm.T - 1) / dm.T;
        const int64_t rg_allow = rows_ok ? std::min<int64_t>({md::kMaxRowGroups, dm.LHkv / md::kMinGroupRows,
                                                              dm.n_wg / std::max<int64_t>(cap_units, 1)})
                                         : 1;
        auto pick = [&](int64_t u) -> int {
            if (u <= 0 || 2 * u >= dm.n_wg) return 1;
            return (int)std::max<int64_t>(1, std::min<int64_t>(rg_allow, dm.n_wg / u));
        };
        rg_first = pick(first);
        rg_steady = pick(steady);
        // the row-group instantiation, when a step will use it, must hold
        // the same grid as the plain one
        if (std::max(rg_first, rg_steady) > 1) {
            int32_t seen[2] = {0, 0};
            bool held = false;
            if (md::launch_attend_check(dm, probe, dm.n_wg, 2, hs) != hipSuccess ||
                hipMemcpyAsync(seen, probe, sizeof(seen), hipMemcpyDeviceToHost, hs) != hipSuccess ||
                hipStreamSynchronize(hs) != hipSuccess) {
                (void)hipGetLastError();
            } else {
                held = seen[1] >= dm.n_wg;
            }
            if (!held) rg_first = rg_steady = 1;
        }
        // Units on every row pay off from half the grid on; row groups, whose
        // units walk few rows, from a quarter (measured on batches of
        // 1,700-token sessions: 8 sessions, 144 units of nine groups, 49.5
        // against 55.5 us per step on the multi-kernel path; 4 sessions, 72
        // units, 46.8 against 44.7 us).
        auto fills = [&](int64_t u, int rg) { return (rg > 1 ? 4 : 2) * u * rg >= dm.n_wg; };
        if (!(cfg->flags & MD_FLAG_FUSED)) {
            fused_first = fills(first, rg_first);
            fused_steady = fills(steady, rg_steady);
        }
        if (!fused_first) rg_first = 1;
        if (!fused_steady) rg_steady = 1;
    }
    free_probe();
    dm.rg_max = std::max(rg_first, rg_steady);
    if (dm.fused) dm.U_cap *= dm.rg_max;
    dm.multi = dm.spill || !fused_first || !fused_steady;

    const size_t bytes = md::scratch_bytes(dm);
    if (use_static && bytes > md::kStaticScratchBytes) return MD_E_TOO_LARGE;
    md_handle_s* h = use_static ? take_static_handle() : new (std::nothrow) md_handle_s();
    if (h == nullptr) return use_static ? MD_E_TOO_LARGE : MD_E_NOMEM;
    if (!use_static) h->static_slot = -1;
    h->dm = dm;
    h->v = md::View{};
    h->v.k_pool = cv->k_pool;
    h->v.region = cv->region;
    h->v.t_ins = cv->t_ins;
    h->v.t_ref = cv->t_ref;
    h->v.imp = cv->importance;
    h->v.page_table = cv->page_table;
    h->v.page_serial = cv->page_serial;
    h->v.n_pages = cv->n_pages;
    h->v.n_tokens = cv->n_tokens;
    h->v.n_live = dm.aligned ? cv->n_live : cv->n_tokens;
    h->v.page_format = dm.quant ? cv->page_format : nullptr;
    h->v.clock = cv->clock;
    h->v.next_serial = cv->next_serial;
    h->v.budget = cv->budget;
    h->v.free_list = cv->free_list;
    h->v.free_count = cv->free_count;
    h->v.b = rp->base_priority;
    h->v.lam = rp->decay_rate;
    if (dm.H > 0) {
        // the pinned host memory's address on the device
        void* dk = nullptr;
        if (hipHostGetDevicePointer(&dk, cv->host_keys, 0) != hipSuccess) {
            (void)hipGetLastError();
            give_back(h);
            return MD_E_INVALID;
        }
        h->v.host_keys = static_cast<unsigned char*>(dk);
        h->v.off_count = cv->off_count;
        h->v.off_serial = cv->off_serial;
        h->v.off_slot = cv->off_slot;
        h->v.off_region = cv->off_region;
        h->v.off_t_ins = cv->off_t_ins;
        h->v.off_t_ref = cv->off_t_ref;
        h->v.off_imp = cv->off_importance;
        h->v.off_format = cv->off_format;
        h->v.off_score = cv->off_score;
        h->v.off_abar = cv->off_abar;
    }
    h->stream = hs;
    h->device = dev;

    if (use_static) {
        h->scratch = static_base;
    } else if (hipMalloc(&h->scratch, bytes) != hipSuccess) {
        give_back(h);
        return MD_E_NOMEM;
    }
    md::scratch_carve(dm, h->scratch, &h->sc);
    // counters, status, epoch and the tagged unit statistics start at zero
    // (no step's tag is zero); work lists are empty until the first append.
    // The static scratch keeps what its last handle left there: cleared too.
    if (hipMemsetAsync(h->scratch, 0, bytes, hs) != hipSuccess || hipStreamSynchronize(hs) != hipSuccess) {
        if (!use_static) (void)hipFree(h->scratch);
        give_back(h);
        return MD_E_HIP;
    }
    h->logits_blocks = 3 * n_cu;
    h->mass_blocks = 4 * n_cu;
    h->score_blocks = 2 * n_cu;
    h->have_step = false;
    h->last_step = 0;
    h->fused_first = fused_first;
    h->fused_steady = fused_steady;
    h->rg_first = rg_first;
    h->rg_steady = rg_steady;
    h->observed = 0;
    h->word_tag = 0;
    h->phase = kNone;
    h->sel_serial = nullptr;
    h->sel_count = nullptr;
    h->profile_mask = 0;
    *out = h;
    return MD_OK;
}

md_status md_init(const md_config* cfg, const md_region_params* rp, const md_cache_view* cv,
                  void* stream, md_handle* out) {
    return init_handle(cfg, rp, cv, stream, out, false);
}

md_status md_init_static(const md_config* cfg, const md_region_params* rp, const md_cache_view* cv,
                         void* stream, md_handle* out) {
    return init_handle(cfg, rp, cv, stream, out, true);
}

md_status md_observe_step(md_handle h, int32_t step, const float* q, const uint16_t* new_k,
                          const uint8_t* new_region, float* abar_out) {
    if (h == nullptr || (q != nullptr && !aligned(q, 16))) return MD_E_INVALID;
    if (new_k != nullptr && (new_region == nullptr || !aligned(new_k, 16))) return MD_E_INVALID;
    if (abar_out != nullptr && !aligned(abar_out, 4)) return MD_E_INVALID;
    if (h->have_step && step != h->last_step + 1) return MD_E_STEP;
    if (hipSetDevice(h->device) != hipSuccess) return MD_E_HIP;
    if (q == nullptr) {
        // a decode step without an observation: the append and the clock only
        if (timed_launch(h, MD_K_APPEND, [&] {
                return md::launch_append(h->dm, h->v, h->sc, new_k, new_region, 0, 0, 1, next_word_tag(h),
                                         h->stream); }) !=
            hipSuccess)
            return MD_E_HIP;
        h->have_step = true;
        h->last_step = step;
        h->phase = kNone;
        h->sel_serial = h->sel_count = nullptr;
        return MD_OK;
    }
    const bool fused = h->observed == 0 ? h->fused_first : h->fused_steady;
    const int rg = fused ? (h->observed == 0 ? h->rg_first : h->rg_steady) : 1;
    hipError_t e = timed_launch(h, MD_K_APPEND, [&] {
        return md::launch_append(h->dm, h->v, h->sc, new_k, new_region, fused ? 1 : 0, 1, rg, next_word_tag(h),
                                 h->stream); });
    // On a fused step, sessions that fit one pass of the fused kernel run
    // there; the others (only possible when a session may outgrow n_wg * T
    // tokens) take the three-kernel path with the logits in HBM, which on
    // the other steps observes every session.
    const bool multi = !fused || h->dm.spill;
    if (e == hipSuccess && fused)
        e = timed_launch_ev(h, MD_K_ATTEND, !h->dm.coop, [&](hipEvent_t t0, hipEvent_t t1) {
            return md::launch_attend(h->dm, h->v, h->sc, q, abar_out, rg, h->stream, t0, t1); });
    if (e == hipSuccess && multi) e = timed_launch(h, MD_K_LOGITS, [&] {
        return md::launch_logits(h->dm, h->v, h->sc, q, h->logits_blocks, h->stream); });
    // Sessions of at most kFoldChunks chunks: the mass kernel works out the
    // row statistics itself (the offload tier reads them, so it keeps the
    // separate kernel).
    const bool fold = h->dm.max_chunks <= md::kFoldChunks && h->dm.H == 0;
    if (e == hipSuccess && multi && !fold) e = timed_launch(h, MD_K_ROWSTATS, [&] {
        return md::launch_rowstats(h->dm, h->sc, h->stream); });
    if (e == hipSuccess && multi) e = timed_launch(h, MD_K_MASS, [&] {
        return md::launch_mass(h->dm, h->v, h->sc, abar_out, h->mass_blocks, fold, h->stream); });
    if (e == hipSuccess && h->dm.H > 0) e = md::launch_recall(h->dm, h->v, h->sc, q, abar_out, h->stream);
    if (e != hipSuccess) return MD_E_HIP;
    h->observed += 1;
    h->have_step = true;
    h->last_step = step;
    h->phase = kObserved;
    h->sel_serial = h->sel_count = nullptr;
    return MD_OK;
}

md_status md_score_pages(md_handle h, float* page_score, float* token_score) {
    if (h == nullptr) return MD_E_INVALID;
    if ((page_score != nullptr && !aligned(page_score, 4)) ||
        (token_score != nullptr && !aligned(token_score, 4)))
        return MD_E_INVALID;
    if (h->phase != kObserved && h->phase != kScored) return MD_E_STATE;
    if (hipSetDevice(h->device) != hipSuccess) return MD_E_HIP;
    // The observation (the fused kernel, or the multi-kernel path's mass
    // kernel) already left every session's page scores in the library's
    // copy; the scoring kernel runs again only to fill the caller's outputs.
    const bool needed = page_score != nullptr || token_score != nullptr;
    if (needed && timed_launch(h, MD_K_SCORE, [&] {
            return md::launch_score(h->dm, h->v, h->sc, page_score, token_score, h->score_blocks,
                                    h->stream); }) != hipSuccess)
        return MD_E_HIP;
    h->phase = kScored;
    return MD_OK;
}

md_status md_select_evict(md_handle h, int32_t* evict_serial, int32_t* evict_count, uint8_t* infeasible) {
    if (h == nullptr || evict_serial == nullptr || evict_count == nullptr || infeasible == nullptr)
        return MD_E_INVALID;
    if (!aligned(evict_serial, 4) || !aligned(evict_count, 4)) return MD_E_INVALID;
    if (h->phase != kScored) return MD_E_STATE;
    if (hipSetDevice(h->device) != hipSuccess) return MD_E_HIP;
    if (timed_launch(h, MD_K_SELECT, [&] {
            return md::launch_select(h->dm, h->v, h->sc, evict_serial, evict_count, infeasible,
                                     h->stream); }) != hipSuccess)
        return MD_E_HIP;
    h->sel_serial = evict_serial;
    h->sel_count = evict_count;
    return MD_OK;
}

md_status md_compact(md_handle h, const int32_t* evict_serial, const int32_t* evict_count) {
    if (h == nullptr || ((evict_serial == nullptr) != (evict_count == nullptr))) return MD_E_INVALID;
    if (h->phase == kNone) return MD_E_STATE;
    const int trusted = evict_serial == nullptr ? 1 : 0;
    if (evict_serial == nullptr) {   // the selection of this step
        if (h->sel_serial == nullptr || h->phase != kScored) return MD_E_STATE;
        evict_serial = h->sel_serial;
        evict_count = h->sel_count;
    }
    if (!aligned(evict_serial, 4) || !aligned(evict_count, 4)) return MD_E_INVALID;
    if (h->dm.quant && h->phase != kScored) return MD_E_STATE;   // the tier needs this step's scores
    if (hipSetDevice(h->device) != hipSuccess) return MD_E_HIP;
    if (h->dm.H > 0 && h->phase != kScored) return MD_E_STATE;   // the tier needs this step's scores
    if (h->dm.H > 0 &&
        md::launch_offload(h->dm, h->v, h->sc, evict_serial, evict_count, h->stream) != hipSuccess)
        return MD_E_HIP;
    if (h->dm.quant &&
        md::launch_quant(h->dm, h->v, h->sc, evict_serial, evict_count, h->stream) != hipSuccess)
        return MD_E_HIP;
    if (timed_launch(h, MD_K_COMPACT, [&] {
            return md::launch_compact(h->dm, h->v, h->sc, evict_serial, evict_count, trusted, h->stream); }) !=
        hipSuccess)
        return MD_E_HIP;
    h->phase = kCompacted;
    h->sel_serial = h->sel_count = nullptr;
    return MD_OK;
}

md_status md_select_compact(md_handle h, int32_t* evict_serial, int32_t* evict_count, uint8_t* infeasible) {
    if (h == nullptr || evict_serial == nullptr || evict_count == nullptr || infeasible == nullptr)
        return MD_E_INVALID;
    if (!aligned(evict_serial, 4) || !aligned(evict_count, 4)) return MD_E_INVALID;
    if (h->phase != kScored) return MD_E_STATE;
    if (h->dm.quant || h->dm.H > 0) {   // the tiers run between the selection and the compaction
        const md_status st = md_select_evict(h, evict_serial, evict_count, infeasible);
        return st != MD_OK ? st : md_compact(h, nullptr, nullptr);
    }
    if (hipSetDevice(h->device) != hipSuccess) return MD_E_HIP;
    const uint32_t tag = next_word_tag(h);
    if (timed_launch(h, MD_K_EVICT, [&] {
            return md::launch_evict(h->dm, h->v, h->sc, evict_serial, evict_count, infeasible, tag,
                                    h->stream); }) != hipSuccess)
        return MD_E_HIP;
    h->phase = kCompacted;
    h->sel_serial = h->sel_count = nullptr;
    return MD_OK;
}

md_status md_read_device_status(md_handle h, int32_t* host_out) {
    if (h == nullptr || host_out == nullptr) return MD_E_INVALID;
    if (hipSetDevice(h->device) != hipSuccess) return MD_E_HIP;
    int32_t v[2] = {0, 0};   // the status word and the warning word next to it
    if (hipMemcpyAsync(v, h->sc.status, sizeof(v), hipMemcpyDeviceToHost, h->stream) != hipSuccess ||
        hipMemsetAsync(h->sc.status, 0, sizeof(v), h->stream) != hipSuccess ||
        hipStreamSynchronize(h->stream) != hipSuccess)
        return MD_E_HIP;
    *host_out = v[0];
    return (v[1] & 1) ? MD_W_BUDGET_INFEASIBLE : MD_OK;
}

md_status md_profile_enable(md_handle h, uint32_t kernel_mask) {
    if (h == nullptr || (kernel_mask >> MD_K_COUNT) != 0) return MD_E_INVALID;
    h->profile_mask = kernel_mask;
    return MD_OK;
}

md_status md_profile_read(md_handle h, int32_t kernel, double* total_ms, int64_t* launches) {
    if (h == nullptr || total_ms == nullptr || launches == nullptr || kernel < 0 || kernel >= MD_K_COUNT)
        return MD_E_INVALID;
    if (hipSetDevice(h->device) != hipSuccess || hipStreamSynchronize(h->stream) != hipSuccess)
        return MD_E_HIP;
    double sum = 0.0;
    md_status st = MD_OK;
    for (auto& t : h->pending[kernel]) {
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, t.start, t.stop) != hipSuccess) st = MD_E_HIP;
        sum += ms;
        h->spare.push_back(t);
    }
    *launches = (int64_t)h->pending[kernel].size();
    h->pending[kernel].clear();
    *total_ms = sum;
    return st;
}

md_status md_calib_accumulate(md_handle h, const float* abar, int32_t bucket_steps, int32_t n_buckets,
                              uint64_t* mass_fx, uint64_t* count, uint64_t* age_sum) {
    if (h == nullptr || abar == nullptr || mass_fx == nullptr || count == nullptr || age_sum == nullptr)
        return MD_E_INVALID;
    if (bucket_steps < 1 || n_buckets < 1 || (int64_t)n_buckets * h->dm.n_regions > (1 << 20))
        return MD_E_INVALID;
    if (!aligned(abar, 4) || !aligned(mass_fx, 8) || !aligned(count, 8) || !aligned(age_sum, 8))
        return MD_E_INVALID;
    if (h->phase == kNone) return MD_E_STATE;
    if (hipSetDevice(h->device) != hipSuccess) return MD_E_HIP;
    if (md::launch_calib(h->dm, h->v, h->sc, abar, bucket_steps, n_buckets,
                         reinterpret_cast<unsigned long long*>(mass_fx),
                         reinterpret_cast<unsigned long long*>(count),
                         reinterpret_cast<unsigned long long*>(age_sum), h->stream) != hipSuccess)
        return MD_E_HIP;
    return MD_OK;
}

md_status md_calib_fit(const uint64_t* mass_fx, const uint64_t* count, const uint64_t* age_sum,
                       int32_t n_sessions, int32_t n_regions, int32_t n_buckets, double* lambda_hat,
                       double* log_c) {
    if (mass_fx == nullptr || count == nullptr || age_sum == nullptr || lambda_hat == nullptr ||
        log_c == nullptr || n_sessions < 1 || n_regions < 1 || n_buckets < 1)
        return MD_E_INVALID;
    const double unit = 1.0 / 1099511627776.0;   // 2^-40
    for (int r = 0; r < n_regions; ++r) {
        // per bucket: weight = observations, x = their mean age, y = log of
        // their mean mass (buckets without observations or mass left out)
        std::vector<double> w, x, y;
        for (int b = 0; b < n_buckets; ++b) {
            double m = 0.0, n = 0.0, a = 0.0;
            for (int s = 0; s < n_sessions; ++s) {
                const size_t i = ((size_t)s * n_regions + r) * n_buckets + b;
                m += (double)mass_fx[i] * unit;
                n += (double)count[i];
                a += (double)age_sum[i];
            }
            if (n > 0.0 && m > 0.0) {
                w.push_back(n);
                x.push_back(a / n);
                y.push_back(log(m / n));
            }
        }
        lambda_hat[r] = log_c[r] = NAN;
        if (w.size() < 2) continue;
        double sw = 0.0, sx = 0.0, sy = 0.0;
        for (size_t i = 0; i < w.size(); ++i) {
            sw += w[i];
            sx += w[i] * x[i];
            sy += w[i] * y[i];
        }
        const double xm = sx / sw, ym = sy / sw;
        double sxx = 0.0, sxy = 0.0;
        for (size_t i = 0; i < w.size(); ++i) {
            sxx += w[i] * (x[i] - xm) * (x[i] - xm);
            sxy += w[i] * (x[i] - xm) * (y[i] - ym);
        }
        if (sxx == 0.0) continue;
        const double slope = sxy / sxx;
        lambda_hat[r] = -slope;
        log_c[r] = ym - slope * xm;
    }
    return MD_OK;
}

md_status md_read_counters(md_handle h, int64_t* out) {
    if (h == nullptr || out == nullptr) return MD_E_INVALID;
    if (hipSetDevice(h->device) != hipSuccess) return MD_E_HIP;
    unsigned long long v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (hipMemcpyAsync(v, h->sc.counters, sizeof(v), hipMemcpyDeviceToHost, h->stream) != hipSuccess ||
        hipStreamSynchronize(h->stream) != hipSuccess)
        return MD_E_HIP;
    for (int i = 0; i < 8; ++i) out[i] = (int64_t)v[i];
    return MD_OK;
}

md_status md_kernel_config(md_handle h, int32_t* out) {
    if (h == nullptr || out == nullptr) return MD_E_INVALID;
    out[0] = h->dm.fused;
    out[1] = h->dm.spill;
    out[2] = h->dm.fused ? h->dm.T : 0;
    out[3] = h->dm.n_wg;
    out[4] = h->fused_first ? 1 : 0;
    out[5] = h->fused_steady ? 1 : 0;
    out[6] = h->rg_first;
    out[7] = h->rg_steady;
    return MD_OK;
}

md_status md_destroy(md_handle h) {
    if (h == nullptr) return MD_E_INVALID;
    md_status st = MD_OK;
    if (hipSetDevice(h->device) != hipSuccess || hipStreamSynchronize(h->stream) != hipSuccess) st = MD_E_HIP;
    release_events(h);
    if (h->static_slot < 0 && hipFree(h->scratch) != hipSuccess) st = MD_E_HIP;
    give_back(h);
    return st;
}

}  // extern "C"
