/*
 * memdecay.h — C ABI of the MemDecay retention hot path on one AMD Instinct
 * MI355X (gfx950).
 *
 * MemDecay ("Region-Aware KV Cache Eviction for Efficient LLM Agent
 * Inference", Sec. III) keeps, for every cached token i of an agent
 * session, a region label r(i), an insertion step, an attention importance
 * a_i (Eq. 2) and a refresh clock t_ref_i (Eq. 3).  At each observation
 * step it scores tokens with s_i = b_r exp(-lambda_r (t - t_ref_i)) + alpha
 * a_i (Eq. 4), averages scores per page (Eq. 5) and, when the session holds
 * more than its budget B, evicts non-pinned pages in ascending page score
 * until the budget holds (Sec. III-D, Alg. 1).  This library runs one such
 * step per call sequence
 *
 *     md_observe_step  ->  md_score_pages  ->  md_select_evict  ->  md_compact
 *
 * (the last two also as one call, md_select_compact)
 *
 * over a batch of independent sessions whose keys live in a paged bf16 pool.
 *
 * Conventions for every entry point
 * ---------------------------------
 *  * All array arguments are DEVICE pointers into memory the caller owns
 *    (allocated with hipMalloc or by a framework on the same device).  The
 *    library never frees them.  Only md_init's struct arguments and the
 *    host_out of md_read_device_status are host pointers.
 *  * Every call enqueues work on the stream given to md_init and returns
 *    without synchronising, except md_init (which validates the region tables
 *    on the host) and md_read_device_status.
 *  * Negative return values are errors detected on the host before anything
 *    was enqueued; the session state is unchanged.  Conditions only the
 *    device can see (free list empty, non-finite query) set bits in a device
 *    status word read by md_read_device_status.  Positive values are
 *    warnings (MD_W_*).
 *  * A handle is not thread-safe; calls on one handle must be serialised.
 *  * Every result is deterministic, the physical page ids included: an
 *    append takes pages off the free list in session order, and md_compact
 *    pushes the freed ids in (session, serial) order.
 *
 * Layouts (S = max_sessions, NP = n_phys_pages, P = page_size, MP = max_pages)
 *  k_pool       uint16 bf16 bits [NP][L][Hkv][P/16][d/8][16][8]   keys of each
 *               physical page: for each (layer, KV head), blocks of 16 tokens,
 *               each block holding dims 8b .. 8b+7 of its 16 tokens together
 *               (block-interleaved, so that the attention kernels read 1 KiB
 *               contiguous per load); element (t, e) of a (page, l, kv) tile
 *               sits at (t & ~15) * d + (e / 8) * 128 + (t % 16) * 8 + e % 8
 *  region       uint8  [NP][P]   region code of each slot
 *  t_ins, t_ref int32  [NP][P]   insertion step, refresh clock of each slot
 *  importance   float  [NP][P]   a_i of each slot
 *  page_table   int32  [S][MP]   physical page ids in logical order
 *  page_serial  int32  [S][MP]   opening serial of each listed page (ascending)
 *  n_pages, n_tokens, clock, next_serial, budget   int32 [S]
 *  free_list    int32  [NP]      stack of free physical ids; free_count int32 [1]
 *  n_live       int32  [S]       tokens of each session (region-aligned pages only)
 * Every page of a session except the last has all P slots in use; the last
 * has n_tokens - (n_pages - 1) * P.  A slot in use holds a token, except with
 * MD_FLAG_REGION_ALIGNED: there the slots of a page after its last token,
 * left unused when the page was closed at a region boundary, are holes
 * (region code MD_REGION_HOLE), n_tokens counts them with the tokens, and
 * n_live counts the tokens alone.
 * Quantised pages (quant_threshold > 0, page_format[p] = 1): each 16-token
 * block of a (layer, KV head) tile keeps, in the first 2 KiB of its 4 KiB,
 * FP8 E4M3 codes c (OCP format: bias 7, no infinities) with key = s * c, and
 * its scale s as float32 in bytes 2048 .. 2051 (repeated in 2052 .. 2063);
 * the code of token t (0..15) and dim e
 * sits at byte 1024 (e / 64) + 16 (t + 16 ((e / 8) % 4)) + 8 ((e / 32) % 2)
 * + e % 8.  Region codes follow the paper's label
 * list: system 0, plan 1, user 2, tool_in 3, tool_out 4, retrieval 5,
 * scratchpad 6.
 */
#ifndef MEMDECAY_H
#define MEMDECAY_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MD_ABI_VERSION 10

typedef int32_t md_status;

enum {
    MD_OK = 0,
    MD_E_INVALID = -1,      /* null or misaligned pointer, bad value            */
    MD_E_UNSUPPORTED = -2,  /* shape outside what the kernels are built for     */
    MD_E_STEP = -3,         /* step did not advance by exactly one              */
    MD_E_HIP = -4,          /* a HIP runtime call failed                        */
    MD_E_STATE = -5,        /* call out of order (e.g. select before score)     */
    MD_E_NOMEM = -6,        /* scratch allocation failed in md_init             */
    MD_E_TOO_LARGE = -7,    /* md_init_static: the scratch exceeds its static   */
                            /* array, or every static handle is in use          */
    MD_W_BUDGET_INFEASIBLE = 1  /* warning (md_read_device_status): some        */
                            /* selection found a session whose pinned tokens   */
                            /* alone exceed its budget (Eq. 1 has no feasible  */
                            /* set); its infeasible flag says which            */
};

/* Bits of the device status word. */
#define MD_DEV_CAPACITY   0x1   /* free list empty or page table full at append */
#define MD_DEV_NONFINITE  0x2   /* NaN or infinity in a decode query: the       */
                                /* session's step is void (see below)          */
#define MD_DEV_BAD_EVICT  0x4   /* md_compact got a serial the session lacks    */
#define MD_DEV_CORRUPT    0x8   /* a session's counters, page table or region   */
                                /* codes are out of range; the session is      */
                                /* skipped for the step                         */
#define MD_DEV_TIMEOUT    0x10  /* a bounded wait between the workgroups of the */
                                /* fused observation kernel ran out; the step's */
                                /* attention mass is not valid                  */
/* A void step.  A session whose decode query is not finite, or whose
 * workgroups of the fused kernel ran out of time, takes no part in the
 * step's selection (evict_count 0), compaction or quantisation, and its
 * tokens keep their importance and refresh clocks (on a time-out, the
 * workgroups that did complete their share of the session's tokens have
 * updated those tokens).  The append and the clock advance stand. */

/* Bits of md_config.flags. */
#define MD_FLAG_NO_FUSED  0x1   /* observe every session with the multi-kernel  */
                                /* path (logits through HBM) instead of the     */
                                /* fused one; results agree to rounding         */
#define MD_FLAG_NORM_ATTENTION 0x4  /* score the attention term against the */
                                /* uniform attention level, as Sec. IV-D        */
                                /* proposes: alpha * |K_t| * a_i in Eq. 4, with */
                                /* |K_t| the session's tokens after the append  */
#define MD_FLAG_REGION_ALIGNED 0x8  /* region-aligned pages (the allocator   */
                                /* variant of Sec. III-D): an appended token    */
                                /* opens a fresh page also when its region      */
                                /* differs from that of the session's last      */
                                /* token, and the last page's unused slots      */
                                /* become holes; needs md_cache_view.n_live     */
#define MD_FLAG_COOPERATIVE 0x10 /* launch the fused observation kernel as a  */
                                /* cooperative launch, which the runtime keeps  */
                                /* from sharing the device with other work; for */
                                /* callers that run kernels on other streams or */
                                /* processes of the same GPU at the same time.  */
                                /* By default it is an ordinary launch (15-20   */
                                /* us less per step): md_init checks that all   */
                                /* its workgroups are resident together on an   */
                                /* idle device, and work on other streams that  */
                                /* takes CUs while it runs can make its bounded */
                                /* waits run out (MD_DEV_TIMEOUT, a void step   */
                                /* for the sessions affected; never a hang)     */
#define MD_REGION_HOLE    0xFF  /* region code of a hole slot                   */
#define MD_FLAG_FUSED     0x2   /* observe on the fused kernel whenever it can  */
                                /* hold the sessions.  With neither flag,       */
                                /* md_init picks the path of the first observe  */
                                /* and of the later ones from the cache's sizes */
                                /* and budgets at init: the fused kernel walks  */
                                /* the layers in order, so for small caches the */
                                /* multi-kernel path, parallel over layers, is  */
                                /* faster                                       */
#define MD_FLAG_NO_ROW_GROUPS 0x20 /* keep every fused unit on all L Hkv rows. */
                                /* By default, on plain pages with one query   */
                                /* per observation, a step whose units would   */
                                /* fill less than half of the fused kernel's   */
                                /* grid splits each unit's rows into up to 16  */
                                /* groups of at least 8 rows, one workgroup    */
                                /* each, whose partial masses (over disjoint   */
                                /* rows of Sec. III-C's mean) are added in a   */
                                /* fixed order; results agree to rounding      */

typedef struct md_config {
    int32_t n_layers;           /* L                                              */
    int32_t n_q_heads;          /* Hq, a multiple of Hkv, Hq/Hkv <= 16            */
    int32_t n_kv_heads;         /* Hkv                                            */
    int32_t head_dim;           /* d; must be 128                                 */
    int32_t page_size;          /* P; 16 or 64                                    */
    int32_t max_sessions;       /* S, 1..1024                                     */
    int32_t max_pages;          /* MP, page-table capacity per session            */
    int32_t n_phys_pages;       /* NP, pages in the pool                          */
    int32_t n_regions;          /* number of region codes, 1..32 (7 in the paper) */
    uint32_t pinned_region_mask;/* bit r set => region r is pinned (Sec. III-A)   */
    float rho;                  /* EWMA smoothing, 0 <= rho < 1 (Eq. 2)           */
    float alpha;                /* attention weight, alpha >= 0 (Eq. 4)           */
    float tau_scale;            /* tau = tau_scale / |K_t| (Eq. 3's scaled form)  */
    int32_t flags;              /* MD_FLAG_* bits; other bits must be 0           */
    int32_t window;             /* W >= 1 decode queries per observation, with    */
                                /* (Hq/Hkv) W <= 16 and L Hq W <= 1024 (Sec.      */
                                /* III-C); both observation paths take W > 1 on   */
                                /* every page layout and tier                     */
    float quant_threshold;      /* quantised tier (Sec. III-E): md_compact turns  */
                                /* pages scoring below it into 8-bit codes; 0 =   */
                                /* off, +INFINITY = every eligible page           */
    int32_t offload_pages;      /* offload tier (Sec. III-E): host-memory pages   */
                                /* per session, 0..64; 0 = off.  Needs window 1   */
                                /* and plain pages (MD_E_UNSUPPORTED otherwise)   */
    float drop_threshold;       /* offload tier: pages scoring below it are       */
                                /* dropped, not kept in host memory (>= 0)        */
} md_config;

/* Region priors (Sec. III-B): b_r >= 0 and lambda_r >= 0 per session and
 * region, float32 device arrays [S][n_regions].  Read at every step. */
typedef struct md_region_params {
    const float* base_priority;  /* b      */
    const float* decay_rate;     /* lambda */
} md_region_params;

typedef struct md_cache_view {
    uint16_t* k_pool;
    uint8_t*  region;
    int32_t*  t_ins;
    int32_t*  t_ref;
    float*    importance;
    int32_t*  page_table;
    int32_t*  page_serial;
    int32_t*  n_pages;
    int32_t*  n_tokens;
    int32_t*  clock;
    int32_t*  next_serial;
    int32_t*  budget;
    int32_t*  free_list;
    int32_t*  free_count;
    int32_t*  n_live;     /* MD_FLAG_REGION_ALIGNED: |K_t| per session; else   */
                          /* ignored (may be NULL: |K_t| is n_tokens)          */
    uint8_t*  page_format;/* quant_threshold > 0: [NP], 0 = bf16 keys, 1 =     */
                          /* quantised; else ignored (may be NULL)             */
    /* Offload tier (offload_pages = H > 0; else ignored, may be NULL).  The   */
    /* pages in host memory of session s are listed in entries 0 .. count-1 of */
    /* row s, serials ascending; each sits in a host slot 0 .. H-1, which      */
    /* indexes the keys and the per-token state.  The caller zeroes off_count; */
    /* the library maintains the rest.                                         */
    void*     host_keys;  /* PINNED HOST memory from hipHostMalloc, 16-byte    */
                          /* aligned: [S][H][L Hkv P d] bf16 bits, each slot a  */
                          /* page in the pool's page layout (codes and scales   */
                          /* for a quantised page)                             */
    int32_t*  off_count;  /* [S]                                               */
    int32_t*  off_serial; /* [S][H] serials of the listed pages, ascending     */
    int32_t*  off_slot;   /* [S][H] host slot of each listed page              */
    uint8_t*  off_region; /* [S][H][P] per host slot and token                 */
    int32_t*  off_t_ins;  /* [S][H][P]                                         */
    int32_t*  off_t_ref;  /* [S][H][P]                                         */
    float*    off_importance; /* [S][H][P]                                     */
    uint8_t*  off_format; /* [S][H] per host slot: 1 = quantised keys          */
    float*    off_score;  /* [S][H] page score of each listed page at the last */
                          /* observation (written by the library)              */
    float*    off_abar;   /* [S][H][P] the last observation's mass of each     */
                          /* host-memory token (written by the library)        */
} md_cache_view;

typedef struct md_handle_s* md_handle;

/* Library ABI version (MD_ABI_VERSION of the build). */
int32_t md_abi_version(void);

/* Text for a status code (static storage; never NULL). */
const char* md_status_str(md_status s);

/*
 * md_init — validate the configuration and buffers, allocate the library's
 * own scratch (attention logits of one step, softmax statistics, page scores,
 * work lists; sized from cfg), and bind everything to `stream` (a
 * hipStream_t; NULL = the null stream) on the current device.
 * Copies the region tables to the host once to check b >= 0, lambda >= 0 and
 * finiteness (Sec. III-B).  On success *out holds a new handle; on failure
 * *out is NULL and nothing is allocated.
 */
md_status md_init(const md_config* cfg, const md_region_params* rp,
                  const md_cache_view* cv, void* stream, md_handle* out);

/*
 * md_init_static — md_init that allocates nothing, for callers that cannot
 * allocate memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The handle's scratch is a file-scope
 * device array of 128 MiB inside the library instead of an allocation: one
 * array per device, held by the device from the library's first use on it
 * until the process ends.  The scratch a configuration needs is mostly the
 * fused kernel's statistics, 16 bytes per softmax row (L Hq W) and 256-token
 * unit of the pool, plus, when the multi-kernel path can run, the logits of
 * every pool slot (4 L Hq W bytes each); a configuration that needs more than
 * 128 MiB gets MD_E_TOO_LARGE.  The handle itself is one of 16 static slots
 * (MD_E_TOO_LARGE when all are taken; md_destroy gives it back).
 * md_init_static clears the part of the array the handle uses (the array
 * keeps whatever the previous static handle left there).  Every static
 * handle on a device uses that device's one array, so two static handles
 * alive on one device at once overwrite each other's scratch and their calls
 * race: keep one static handle per device at a time.  Arguments, checks,
 * synchronisation and the calls that follow are those of md_init.
 */
md_status md_init_static(const md_config* cfg, const md_region_params* rp, const md_cache_view* cv,
                         void* stream, md_handle* out);

/*
 * md_observe_step — one decode step; with q given, also an observation step
 * (Alg. 1's importance and refresh updates; attention is sampled every k-th decode step with
 * a window of the W latest decode queries, Sec. III-C):
 *   append: each session's clock advances, t <- t + 1.  If new_k is not NULL
 *     the step's token joins the session's last page, or a page popped from
 *     the free list when the last page is full, with region new_region[s],
 *     t_ins = t_ref = t, a = 0 (Fig. 1, the decode engine's append).  With
 *     MD_FLAG_REGION_ALIGNED the token also opens a fresh page when its
 *     region differs from the last token's; the old page's unused slots
 *     become holes (region MD_REGION_HOLE, t_ins = t_ref = 0, a = 0).
 *     Holes take no part in anything below.
 *   attention mass: for every cached token i, A_i = (1 / (L Hq W)) sum over
 *     layers l, query heads h and window queries w of
 *     softmax_i(q_{w,l,h} . k_{l,h/G,i} / sqrt(d)), the softmax of window
 *     query w running over the session's cached tokens inserted at or
 *     before its step t - (W - 1 - w) (Sec. III-C).  With W = 1: every
 *     cached token.
 *   EWMA (Eq. 2): a_i <- rho a_i + (1 - rho) A_i for every cached token.
 *   refresh (Eq. 3): t_ref_i <- t when A_i >= tau_scale / |K_t|, |K_t| the
 *     session's token count after the append (n_live with region-aligned
 *     pages, n_tokens otherwise).
 *   offload tier (offload_pages > 0; Sec. III-E's second tier): every token
 *     of a page in host memory is observed with the same query, its keys read
 *     over the host link: A_i = the mean over rows of its weight
 *     exp(x_i - M_r) / Lambda_r next to the cached tokens (M_r, Lambda_r:
 *     row r's maximum and sum over the cached tokens, which keep their
 *     masses; 0 without cached tokens); EWMA, refresh (same tau), token and
 *     page scores as for a cached token (off_importance, off_t_ref,
 *     off_abar, off_score).  A page with a token refreshed now is recalled:
 *     a device page comes off the free list (sessions in order), the keys
 *     and token state come back, and the page rejoins the page table in
 *     serial order, so this step's selection counts it.
 * q:          float32 [S][W][L][Hq][d] decode queries of steps t - W + 1 .. t,
 *             oldest first (device), or NULL for a decode step without an
 *             observation: then only the append and the clock advance run,
 *             and md_score_pages, md_select_evict and md_compact answer
 *             MD_E_STATE until the next observation.
 * new_k:      bf16 bits [S][L][Hkv][d] keys of the appended tokens, or NULL.
 * new_region: uint8 [S] region codes of the appended tokens; required with new_k.
 * abar_out:   optional float32 [NP][P]; receives A_i at each live slot.
 * step:       any value on the first call, then exactly the previous + 1
 *             (MD_E_STEP otherwise, nothing enqueued).
 */
md_status md_observe_step(md_handle h, int32_t step, const float* q,
                          const uint16_t* new_k, const uint8_t* new_region,
                          float* abar_out);

/*
 * md_score_pages — retention scores and page scores (Alg. 1's scoring steps):
 *   s_i = b_{r(i)} exp(-lambda_{r(i)} (t - t_ref_i)) + alpha a_i    (Eq. 4)
 *   S_p = (1/|p|) sum_{i in p} s_i over the page's live tokens      (Eq. 5)
 * Pinned tokens bypass scoring (+INFINITY); a page with any pinned member
 * is pinned and scores +INFINITY.
 * page_score:  optional float32 [S][MP], logical page order.
 * token_score: optional float32 [NP][P] at each live slot.
 * The library keeps its own copy of the page scores for md_select_evict;
 * md_observe_step completes it on either observation path, so a call with
 * both outputs NULL enqueues nothing.
 * Requires md_observe_step since the last md_compact (MD_E_STATE otherwise).
 */
md_status md_score_pages(md_handle h, float* page_score, float* token_score);

/*
 * md_select_evict — budget-aware page eviction (Alg. 1's eviction loop): when a
 * session holds n > B tokens (B = budget[s]; a page counts its tokens, not
 * its holes), the shortest prefix of its
 * non-pinned pages in ascending (S_p, serial) order whose removal leaves
 * n <= B.  If even all non-pinned pages are not enough, all of them are
 * selected and infeasible[s] = 1 (the pinned set alone exceeds B).
 * evict_serial: int32 [S][MP]; row s receives evict_count[s] serials, ascending.
 * evict_count:  int32 [S].   infeasible: uint8 [S].
 * Mutates no session state; may be called again.  Requires md_score_pages
 * since the last md_observe_step.
 */
md_status md_select_evict(md_handle h, int32_t* evict_serial, int32_t* evict_count,
                          uint8_t* infeasible);

/*
 * md_compact — apply an eviction (Sec. III-E: irreversible): remove the
 * listed pages from each session's page table and serial list keeping the
 * order of the rest, update n_pages / n_tokens (and n_live with
 * region-aligned pages), and push the freed physical ids onto the free list
 * in (session, serial) order.
 * evict_serial / evict_count: both NULL to apply this step's selection (the
 * lists of the last md_select_evict since md_observe_step; MD_E_STATE when
 * there was none), or both given, with md_select_evict's layout, to apply
 * other lists (a caller's own choice; one NULL and one not is
 * MD_E_INVALID).  Serials a session does not hold set MD_DEV_BAD_EVICT and
 * are ignored.  Sessions whose step is void are left as they are.
 * Offload tier (offload_pages > 0; Sec. III-E), first: pages in host memory
 * whose score of this step is below drop_threshold are dropped; of the
 * listed pages, those that take no more tokens (all but the last page, or a
 * full last page) and score at least drop_threshold are copied to host
 * memory with their tokens' state, the highest score first (then the older
 * page), while the session has free host slots; the others are dropped.
 * Requires md_score_pages since the last md_observe_step.
 * Quantised tier (quant_threshold > 0; Sec. III-E's first tier): before the
 * compaction, every page that survives, is not pinned, is not the session's
 * last page, is still bf16 and has page score S_p < quant_threshold (the
 * scores of this step's md_score_pages) is quantised in place: per 16-token
 * block and (layer, KV head), s = max|k| / 448 in float32 and c = the E4M3
 * value nearest to the float32 quotient k / s (ties to even, saturating at
 * 448; s = 0, c = 0 for an all-zero block; holes get c = 0), page_format = 1.  Irreversible.  Requires md_score_pages since the
 * last md_observe_step (MD_E_STATE otherwise).
 */
md_status md_compact(md_handle h, const int32_t* evict_serial, const int32_t* evict_count);

/*
 * md_select_compact — md_select_evict followed by md_compact(h, NULL, NULL)
 * (Alg. 1's eviction loop and its application, Sec. III-D and III-E) as one
 * call: the same lists, infeasible flags, page tables, counts and free list
 * as the two calls.  Without a tier (offload_pages = 0, quant_threshold = 0)
 * it is one launch, each session's block selecting and compacting its own
 * pages; with a tier it enqueues the two calls' launches.  For callers that
 * apply the library's own selection without looking at it in between.
 * Arguments, layout and requirements as for md_select_evict.  In the one
 * launch each block finds its session's places on the free list from the
 * counts of the sessions before it, with bounded waits (1 ms); a wait that
 * runs out, possible only while other work holds the compute units, sets
 * MD_DEV_CORRUPT: that session is left as it was (its lists are still
 * written), and the free count is then not updated, so no page can be
 * handed out twice (the pages the other sessions freed are lost to the
 * free list).
 */
md_status md_select_compact(md_handle h, int32_t* evict_serial, int32_t* evict_count, uint8_t* infeasible);

/* Synchronise the stream and copy the device status word to *host_out, then
 * clear it.  Returns MD_W_BUDGET_INFEASIBLE when a selection since the last
 * read found a session whose pinned tokens exceed its budget (the
 * selection itself cannot report it without synchronising), MD_OK
 * otherwise, and MD_E_HIP if the stream reports an error. */
md_status md_read_device_status(md_handle h, int32_t* host_out);

/* Kernel ids for md_profile_enable / md_profile_read. */
enum {
    MD_K_APPEND = 0, MD_K_LOGITS = 1, MD_K_ROWSTATS = 2, MD_K_MASS = 3,
    MD_K_SCORE = 4, MD_K_SELECT = 5, MD_K_COMPACT = 6, MD_K_ATTEND = 7,
    MD_K_EVICT = 8,   /* md_select_compact's one-launch form */
    MD_K_COUNT = 9
};

/* Diagnostics.  md_profile_enable: from now on, time every launch of the
 * kernels whose bit (1 << id) is set in kernel_mask with a pair of hipEvents
 * on the handle's stream (0 turns timing off): the fused observation kernel
 * (ordinary launch) records the pair with its own dispatch, so the pair
 * holds the kernel alone; the others are bracketed by the pair.
 * md_profile_read: synchronise,
 * return the summed duration in milliseconds and the number of timed launches
 * of kernel `kernel` since the last read, and reset them. */
md_status md_profile_enable(md_handle h, uint32_t kernel_mask);
md_status md_profile_read(md_handle h, int32_t kernel, double* total_ms, int64_t* launches);

/* Device-side running totals since md_init, read after synchronising (out:
 * 8 values): out[0] tokens scored (sum over steps and sessions of |K_t|),
 * out[1] steps observed, out[2] pages evicted, out[3] tokens evicted; offload
 * tier: out[4] pages moved to host memory, out[5] pages recalled from it,
 * out[6] pages dropped from it, out[7] host-memory pages observed (each read
 * once over the host link per observation). */
md_status md_read_counters(md_handle h, int64_t* out);

/* How md_init laid out the observation step on this device (out: 8 ints):
 * out[0] 1 when the fused observation kernel is available, out[1] 1 when a
 * session could outgrow one pass of it (those sessions always take the
 * multi-kernel path), out[2] the largest fused unit in tokens, out[3] the
 * fused kernel's workgroups (all resident at once), out[4] 1 when the first
 * md_observe_step runs the fused kernel, out[5] 1 when the later ones do,
 * out[6] and out[7] the row groups of their fused units (1: none; see
 * MD_FLAG_NO_ROW_GROUPS).  Host-only, no device work. */
md_status md_kernel_config(md_handle h, int32_t* out);

/*
 * md_calib_accumulate — region-lifetime statistics for the calibration of
 * the decay rates (Sec. IV-B): adds every token now in the page tables, of
 * every session, to its bin (s, r(i), b), b = (t - t_ins_i) / bucket_steps
 * (ages of n_buckets * bucket_steps steps and more are left out):
 *   mass_fx[s][r][b] += round(A_i * 2^40)   (A_i read from abar at the slot)
 *   count[s][r][b]   += 1
 *   age_sum[s][r][b] += t - t_ins_i
 * abar: float32 [NP][P], e.g. md_observe_step's abar_out of this step.
 * mass_fx, count, age_sum: uint64 [S][n_regions][n_buckets] (device), owned
 * and zeroed by the caller; the integer sums make the result independent of
 * the order of the additions.  Requires an observation since the last
 * md_compact (MD_E_STATE otherwise); enqueued on the handle's stream.
 */
md_status md_calib_accumulate(md_handle h, const float* abar, int32_t bucket_steps, int32_t n_buckets,
                              uint64_t* mass_fx, uint64_t* count, uint64_t* age_sum);

/*
 * md_calib_fit — the log-linear decay of Eq. 6, log A_r(dt) ~ log c_r -
 * lambda_r dt, fitted per region by least squares weighted with each
 * bucket's observation count (Sec. IV-A), on HOST copies of the sums above,
 * added over the n_sessions sessions.  A bucket contributes its mean age and
 * the log of its mean mass; buckets without observations or mass are left
 * out.  Writes lambda_hat[r] and log_c[r] (doubles, n_regions each), NaN for
 * a region with fewer than two usable buckets.  The half-life is
 * ln 2 / lambda_hat (Eq. 7).  Host only, no handle.
 */
md_status md_calib_fit(const uint64_t* mass_fx, const uint64_t* count, const uint64_t* age_sum,
                       int32_t n_sessions, int32_t n_regions, int32_t n_buckets, double* lambda_hat,
                       double* log_c);

/* Release the scratch and the handle (synchronises the stream first). */
md_status md_destroy(md_handle h);

#ifdef __cplusplus
}
#endif

#endif /* MEMDECAY_H */
