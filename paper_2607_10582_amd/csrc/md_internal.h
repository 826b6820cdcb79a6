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

constexpr int kDevCorrupt = MD_DEV_CORRUPT;

struct Dims {
    int L, Hq, Hkv, G, P, Pshift, S, MP, NP, R, LHkv, n_regions, max_chunks;
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
    int32_t* clock;
    int32_t* next_serial;
    int32_t* budget;
    int32_t* free_list;
    int32_t* free_count;
    const float* b;
    const float* lam;
};

struct Scratch {
    float* logits;       // [NP][R][P] base-2 logits of the step (log2(e) q.k / sqrt(d))
    float2* cstats;      // [S][R][max_chunks] (max, sum of 2^(x - max)) per chunk
    float2* rstats;      // [S][R] (row max M, 1 / row sum)
    float* pscore;       // [S][MP] page scores of the step
    int32_t* item_prefix;  // [S + 1] prefix of attention work items (chunks * L * Hkv)
    int32_t* tile_prefix;  // [S + 1] prefix of 64-token tiles
    int32_t* chunks;       // [S] chunks per session (0 for a skipped session)
    int32_t* valid;        // [S] 1 when the session's counters are consistent
    int32_t* done;         // [1] completion counter of the append kernel
    int32_t* status;       // [1] device status word
    unsigned long long* counters;  // [4] tokens scored, steps, pages evicted, tokens evicted
};

size_t scratch_bytes(const Dims& dm);
void scratch_carve(const Dims& dm, void* base, Scratch* sc);

// Launchers; each returns the hipError_t of its launch.
hipError_t launch_append(const Dims& dm, const View& v, const Scratch& sc,
                         const uint16_t* new_k, const uint8_t* new_region, hipStream_t st);
hipError_t launch_logits(const Dims& dm, const View& v, const Scratch& sc, const float* q,
                         int n_blocks, hipStream_t st);
hipError_t launch_rowstats(const Dims& dm, const Scratch& sc, hipStream_t st);
hipError_t launch_mass(const Dims& dm, const View& v, const Scratch& sc, float* abar_out,
                       int n_blocks, hipStream_t st);
hipError_t launch_score(const Dims& dm, const View& v, const Scratch& sc, float* page_score,
                        float* token_score, int n_blocks, hipStream_t st);
hipError_t launch_select(const Dims& dm, const View& v, const Scratch& sc, int32_t* ev_serial,
                         int32_t* ev_count, uint8_t* infeasible, hipStream_t st);
hipError_t launch_compact(const Dims& dm, const View& v, const Scratch& sc,
                          const int32_t* ev_serial, const int32_t* ev_count, hipStream_t st);

}  // namespace md
