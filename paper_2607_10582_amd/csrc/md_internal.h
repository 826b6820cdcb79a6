// Internal declarations shared by the C-ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/memdecay.h"

namespace md {

constexpr int kHeadDim = 128;       // d
constexpr int kChunk = 128;         // tokens per attention work item (8 MFMA row tiles)
constexpr int kTile = 64;           // tokens per mass / score work tile
constexpr int kMaxSessions = 1024;
constexpr int kMaxRows = 1024;      // L * Hq
constexpr int kMaxPages = 8192;     // page-table capacity per session
constexpr int kSelThreads = 1024;   // select / compact block size
constexpr int kPerThread = kMaxPages / kSelThreads;
// Fused observation kernel (k_attend): four waves per workgroup, all doing
// the same job; a unit of work is one session's block of 256 tokens (each
// wave's four tiles of 16 tokens) over every (layer, KV head) row.
constexpr int kAttendPerCu = 2;   // at most two workgroups per CU
inline int attend_threads(int) { return 256; }
inline int attend_unit_tokens(int) { return 256; }
constexpr int kConsumeLag = 7;   // rows a unit runs ahead of the row it normalises
// Row groups: when a step's units fill less than half of the fused grid, each
// unit may cover one of up to kMaxRowGroups ranges of the L * Hkv rows
// (at least kMinGroupRows rows each), the groups' partial masses meeting in
// the unit of the first group.
constexpr int kMaxRowGroups = 16;
constexpr int kMinGroupRows = 8;
constexpr int kRowBufs = kConsumeLag + 1;       // rows of logits held in LDS

constexpr int kFoldChunks = 16;    // multi-kernel path: sessions of at most 2,048 tokens fold their row statistics into the mass kernel
constexpr int kMaxOffload = 64;     // host-tier pages per session at most (one 64-bit slot mask)

constexpr int kDevCorrupt = MD_DEV_CORRUPT;
constexpr int kHole = MD_REGION_HOLE;   // region code of a hole slot (region-aligned pages)

struct Dims {
    int L, Hq, Hkv, G, P, Pshift, S, MP, NP, R, LHkv, n_regions, max_chunks;
    int W;         // window: decode queries per observation (R = L * Hq * W)
    int fused;     // 1: sessions that fit one pass run on k_attend
    int coop;      // 1: k_attend is a cooperative launch (MD_FLAG_COOPERATIVE)
    int spill;     // 1: some session may not fit a pass (the spill kernels run)
    int multi;     // 1: the multi-kernel path runs at some step (its scratch exists)
    int norm_attn; // 1: the attention term of Eq. 4 is alpha * |K_t| * a_i
    int aligned;   // 1: region-aligned pages (hole slots; n_live counts the tokens)
    int quant;     // 1: quantised tier on (pages may hold 8-bit codes)
    float quant_thr;  // quantised tier: pages scoring below it are quantised
    int H;         // offload tier: host-memory pages per session (0: off)
    float drop_thr;   // offload tier: pages scoring below it are dropped
    size_t page_bytes;  // bytes of one page's keys, L * Hkv * P * d * 2
    int n_wg;      // k_attend workgroups (all co-resident)
    int wg_per_cu; // k_attend workgroups per CU (n_wg = wg_per_cu * CUs)
    int lane_cap;  // units one lane of k_attend workgroups holds (one workgroup per CU)
    int T;         // tokens per fused unit (attend_unit_tokens(G))
    int U_cap;     // capacity of the per-step fused unit list
    int rg_max;    // most row groups any step uses (1: none; sizes the partial masses)
    uint32_t pin_mask;
    float rho, alpha, tau_scale;
};

struct View {
    uint16_t* k_pool;
    uint8_t* region;
    int32_t* t_ins;
    int32_t* t_ref;
    float* imp;
    int32_t* page_table;
    int32_t* page_serial;
    int32_t* n_pages;
    int32_t* n_tokens;
    int32_t* n_live;   // [S] tokens |K_t|: the n_tokens array itself unless aligned
    uint8_t* page_format;  // [NP] quantised tier: 1 = the page holds 8-bit codes
    int32_t* clock;
    int32_t* next_serial;
    int32_t* budget;
    int32_t* free_list;
    int32_t* free_count;
    const float* b;
    const float* lam;
    // offload tier (H > 0): the keys of host-memory pages and their
    // per-token state, indexed by (session, host slot)
    unsigned char* host_keys;  // device address of the pinned host memory [S][H][page_bytes]
    int32_t* off_count;        // [S] pages in host memory
    int32_t* off_serial;       // [S][H] their serials, ascending
    int32_t* off_slot;         // [S][H] host slot of each listed page
    uint8_t* off_region;       // [S][H][P] by host slot
    int32_t* off_t_ins;
    int32_t* off_t_ref;
    float* off_imp;
    uint8_t* off_format;       // [S][H] by host slot
    float* off_score;          // [S][H] page score of each listed page
    float* off_abar;           // [S][H][P] by host slot: the step's mass
};

struct Scratch {
    float* logits;       // [NP][R][P] base-2 logits of the step (log2(e) q.k / sqrt(d))
    float2* cstats;      // [S][R][max_chunks] (max, sum of 2^(x - max)) per chunk or fused unit
    float2* rstats;      // [S][R] (row max M, 1 / row sum)
    float* pscore;       // [S][MP] page scores of the step
    int32_t* item_prefix;  // [S + 1] prefix of attention work items (chunks * L * Hkv), spill path
    int32_t* tile_prefix;  // [S + 1] prefix of 64-token tiles, spill path (mass)
    int32_t* score_prefix; // [S + 1] prefix of 64-token tiles, every session (scores)
    int32_t* ustart;       // [S + 1] prefix of fused units over the sessions
    int32_t* plan;         // [1 + 3 (S + 1)]: passes, then (unit tokens, first, end session) per pass
    int32_t* epoch;        // [1] observation counter; tags the fused unit statistics
    unsigned long long* claim;     // [1] lane mode: (first, end) of the sessions no lane has claimed
    unsigned long long* lane_box;  // [kAttendPerCu][S + 1] lane mode: tagged session range of each lane pass
    unsigned long long* ustat;  // [U_cap][R][2] tagged (max, sum) of each fused unit's rows
    unsigned long long* unorm;  // [S][R][2] tagged row normalisers (M, 1 / Lambda) of the fused sessions
    unsigned long long* upart;  // [U_cap][T] row groups: tagged partial masses of each unit's tokens
    int32_t* chunks;       // [S] chunks per session (0 for a skipped session)
    int32_t* valid;        // [S] 1 while the session's step stands: its counters are
                           // consistent, its query finite and no wait of the fused
                           // kernel ran out; 0 leaves it out of selection and compaction
    int32_t* freed;        // [S + 1] pages each session's compaction frees
    int32_t* status;       // [1] device status word
    int32_t* warn;         // [1] warning bits (1: some session's budget was infeasible)
    int32_t* done_compact; // [1] completion counter of the compaction and recall kernels
    unsigned long long* compact_acc;   // [1] the same for its trusted form: blocks done << 40 | gaps
    unsigned long long* app_word;      // [S] append kernel: each session's new counts, tagged
    unsigned long long* ev_word;       // [S] select-and-compact kernel: each session's eviction count, tagged
    unsigned long long* ev_done;       // [S] the same kernel: whether each block applied its selection, tagged
    int32_t* opened;       // [1] pages the recall kernel takes from the free list
    unsigned long long* counters;  // [8] tokens scored, steps, pages evicted, tokens evicted, pages
                                   // offloaded, recalled, dropped from host memory, observed there
    int32_t* recall;       // [S][H] offload tier: the listed page is recalled at this step
    int32_t* rcount;       // [S] pages each session recalls at this step
};

size_t scratch_bytes(const Dims& dm);
void scratch_carve(const Dims& dm, void* base, Scratch* sc);

// md_init_static: the library's scratch in a file-scope device array of this
// size (one per device, held until the process ends) instead of an
// allocation.  static_scratch gives its address on the current device,
// looked up once per device.
constexpr size_t kStaticScratchBytes = (size_t)128 << 20;
hipError_t static_scratch(void** ptr);

// Launchers; each returns the hipError_t of its launch.
// fused: this step observes on the fused kernel (sessions that fit a pass)
// or, when 0, every session on the multi-kernel path.  observe: 0 for a
// decode step without an observation (no work lists, no scored tokens).
// tag: differs from the previous launch's (27 bits used)
constexpr uint32_t kWordTagMask = (1u << 27) - 1;
// Bound of a wait for another block's tagged word (s_memrealtime ticks of
// 10 ns): 50 ms, far beyond any scheduling delay of a running kernel.
constexpr uint64_t kWordWaitTicks = 5000000ull;
// rg: row groups of the step's fused units (1: none)
hipError_t launch_append(const Dims& dm, const View& v, const Scratch& sc,
                         const uint16_t* new_k, const uint8_t* new_region, int fused, int observe,
                         int rg, uint32_t tag, hipStream_t st);
hipError_t launch_logits(const Dims& dm, const View& v, const Scratch& sc, const float* q,
                         int n_blocks, hipStream_t st);
hipError_t launch_rowstats(const Dims& dm, const Scratch& sc, hipStream_t st);
// rg: row groups, as given to the step's append.  t0, t1: when not NULL
// (ordinary launches only), an event pair recorded by the kernel's dispatch
// itself
hipError_t launch_attend(const Dims& dm, const View& v, const Scratch& sc, const float* q,
                         float* abar_out, int rg, hipStream_t st, hipEvent_t t0 = nullptr,
                         hipEvent_t t1 = nullptr);
size_t attend_lds_bytes(int G);
// the instantiation for G MFMA columns (heads per KV head x window), layout,
// tier, window and row groups (> 1: the row-group instantiation)
const void* attend_kernel(int G, int aligned, int quant, int window, int row_groups);
// Launch the fused kernel (the instantiation for rg row groups) in check
// mode with n_wg workgroups: every wave waits (bounded, ~20 ms) until all
// workgroups have arrived; probe[1] receives the fewest arrivals any
// workgroup saw (probe: 2 device ints).
hipError_t launch_attend_check(const Dims& dm, int32_t* probe, int n_wg, int rg, hipStream_t st);
// fold: the mass kernel works out the row statistics itself (no
// launch_rowstats before it; sessions of at most kFoldChunks chunks).  It
// also writes the page scores of the sessions it observes.
hipError_t launch_mass(const Dims& dm, const View& v, const Scratch& sc, float* abar_out,
                       int n_blocks, bool fold, hipStream_t st);
hipError_t launch_score(const Dims& dm, const View& v, const Scratch& sc, float* page_score,
                        float* token_score, int n_blocks, hipStream_t st);
hipError_t launch_select(const Dims& dm, const View& v, const Scratch& sc, int32_t* ev_serial,
                         int32_t* ev_count, uint8_t* infeasible, hipStream_t st);
hipError_t launch_calib(const Dims& dm, const View& v, const Scratch& sc, const float* abar, int bucket_steps,
                        int n_buckets, unsigned long long* mass_fx, unsigned long long* count,
                        unsigned long long* age_sum, hipStream_t st);
// trusted: the lists are the library's own selection of this step
hipError_t launch_evict(const Dims& dm, const View& v, const Scratch& sc, int32_t* ev_serial,
                        int32_t* ev_count, uint8_t* infeasible, uint32_t tag, hipStream_t st);
hipError_t launch_compact(const Dims& dm, const View& v, const Scratch& sc,
                          const int32_t* ev_serial, const int32_t* ev_count, int trusted, hipStream_t st);
// Quantised tier, before the compaction of the same eviction lists.
hipError_t launch_quant(const Dims& dm, const View& v, const Scratch& sc,
                        const int32_t* ev_serial, const int32_t* ev_count, hipStream_t st);
// Offload tier.  At an observation, after the attention: launch_recall
// observes the host-memory pages and recalls those that became relevant
// (q: the step's queries, abar_out: optional masses).  At md_compact,
// before the quantised tier and the compaction: launch_offload drops
// host-memory pages below the threshold and moves leaving pages there.
hipError_t launch_recall(const Dims& dm, const View& v, const Scratch& sc, const float* q, float* abar_out,
                         hipStream_t st);
hipError_t launch_offload(const Dims& dm, const View& v, const Scratch& sc, const int32_t* ev_serial,
                          const int32_t* ev_count, hipStream_t st);

}  // namespace md
