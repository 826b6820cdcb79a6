/* Host-side checks of the C ABI's argument validation and of md_calib_fit,
 * built with AddressSanitizer and UndefinedBehaviorSanitizer together with a
 * host-only build of the library (tests/test_host_sanitizer.py).  Every call
 * below returns before the HIP runtime is touched, so no GPU is needed.
 * Exit status 0 when every call returns what include/memdecay.h promises. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "memdecay.h"

static int fails = 0;

#define EXPECT(call, want)                                                                      \
    do {                                                                                        \
        const md_status got_ = (call);                                                          \
        if (got_ != (want)) {                                                                   \
            fprintf(stderr, "line %d: %s -> %d, expected %d\n", __LINE__, #call, got_, (want)); \
            ++fails;                                                                            \
        }                                                                                       \
    } while (0)

/* A configuration md_init accepts (1.5B attention shape, pages of 16). */
static md_config good_config(void) {
    md_config c;
    memset(&c, 0, sizeof(c));
    c.n_layers = 28;
    c.n_q_heads = 12;
    c.n_kv_heads = 2;
    c.head_dim = 128;
    c.page_size = 16;
    c.max_sessions = 16;
    c.max_pages = 2100;
    c.n_phys_pages = 40000;
    c.n_regions = 7;
    c.pinned_region_mask = 1u;
    c.rho = 0.9f;
    c.alpha = 1.0f;
    c.tau_scale = 2.0f;
    c.flags = 0;
    c.window = 1;
    c.quant_threshold = 0.0f;
    c.offload_pages = 0;
    c.drop_threshold = 0.0f;
    return c;
}

/* Host buffers standing in for the caller's device buffers: validation only
 * looks at the pointers and their alignment. */
static unsigned char* arena;

static md_cache_view good_view(void) {
    md_cache_view v;
    memset(&v, 0, sizeof(v));
    unsigned char* p = arena;
    v.k_pool = (uint16_t*)(p + 0);
    v.region = p + 1024;
    v.t_ins = (int32_t*)(p + 2048);
    v.t_ref = (int32_t*)(p + 3072);
    v.importance = (float*)(p + 4096);
    v.page_table = (int32_t*)(p + 5120);
    v.page_serial = (int32_t*)(p + 6144);
    v.n_pages = (int32_t*)(p + 7168);
    v.n_tokens = (int32_t*)(p + 8192);
    v.clock = (int32_t*)(p + 9216);
    v.next_serial = (int32_t*)(p + 10240);
    v.budget = (int32_t*)(p + 11264);
    v.free_list = (int32_t*)(p + 12288);
    v.free_count = (int32_t*)(p + 13312);
    return v;
}

static void offload_view(md_cache_view* v) {
    unsigned char* p = arena + 16384;
    v->host_keys = p;
    v->off_count = (int32_t*)(p + 1024);
    v->off_serial = (int32_t*)(p + 2048);
    v->off_slot = (int32_t*)(p + 3072);
    v->off_region = p + 4096;
    v->off_t_ins = (int32_t*)(p + 5120);
    v->off_t_ref = (int32_t*)(p + 6144);
    v->off_importance = (float*)(p + 7168);
    v->off_format = p + 8192;
    v->off_score = (float*)(p + 9216);
    v->off_abar = (float*)(p + 10240);
}

static void check_config(md_config c, md_status want, int line) {
    md_cache_view v = good_view();
    if (c.offload_pages > 0) offload_view(&v);
    float b[7 * 16], lam[7 * 16];
    md_region_params rp = {b, lam};
    md_handle h = (md_handle)(uintptr_t)0x1;
    const md_status got = md_init(&c, &rp, &v, NULL, &h);
    if (got != want || h != NULL) {
        fprintf(stderr, "line %d: md_init -> %d (handle %p), expected %d and a NULL handle\n", line, got, (void*)h,
                want);
        ++fails;
    }
    h = (md_handle)(uintptr_t)0x1;
    const md_status got_s = md_init_static(&c, &rp, &v, NULL, &h);
    if (got_s != want || h != NULL) {
        fprintf(stderr, "line %d: md_init_static -> %d, expected %d\n", line, got_s, want);
        ++fails;
    }
}

#define CONFIG_CASE(field_assign, want)           \
    do {                                          \
        md_config c_ = good_config();             \
        field_assign;                             \
        check_config(c_, (want), __LINE__);       \
    } while (0)

static void check_view(md_cache_view v, md_config c, md_status want, int line) {
    float b[7 * 16], lam[7 * 16];
    md_region_params rp = {b, lam};
    md_handle h = NULL;
    const md_status got = md_init(&c, &rp, &v, NULL, &h);
    if (got != want || h != NULL) {
        fprintf(stderr, "line %d: md_init (view) -> %d, expected %d\n", line, got, want);
        ++fails;
    }
}

static void config_cases(void) {
    CONFIG_CASE(c_.flags = 0x100, MD_E_INVALID);
    CONFIG_CASE(c_.flags = MD_FLAG_FUSED | MD_FLAG_NO_FUSED, MD_E_INVALID);
    CONFIG_CASE(c_.offload_pages = -1, MD_E_INVALID);
    CONFIG_CASE(c_.offload_pages = 65, MD_E_INVALID);
    CONFIG_CASE(c_.drop_threshold = NAN, MD_E_INVALID);
    CONFIG_CASE(c_.drop_threshold = -1.0f, MD_E_INVALID);
    CONFIG_CASE((c_.offload_pages = 4, c_.window = 2), MD_E_UNSUPPORTED);
    CONFIG_CASE((c_.offload_pages = 4, c_.flags = MD_FLAG_REGION_ALIGNED), MD_E_UNSUPPORTED);
    CONFIG_CASE(c_.n_layers = 0, MD_E_INVALID);
    CONFIG_CASE(c_.n_kv_heads = 5, MD_E_INVALID);
    CONFIG_CASE(c_.max_sessions = 0, MD_E_INVALID);
    CONFIG_CASE(c_.n_phys_pages = 0, MD_E_INVALID);
    CONFIG_CASE(c_.n_regions = 0, MD_E_INVALID);
    CONFIG_CASE(c_.n_regions = 33, MD_E_INVALID);
    CONFIG_CASE(c_.pinned_region_mask = 1u << 7, MD_E_INVALID);
    CONFIG_CASE(c_.rho = 1.0f, MD_E_INVALID);
    CONFIG_CASE(c_.rho = NAN, MD_E_INVALID);
    CONFIG_CASE(c_.alpha = -0.5f, MD_E_INVALID);
    CONFIG_CASE(c_.alpha = INFINITY, MD_E_INVALID);
    CONFIG_CASE(c_.tau_scale = NAN, MD_E_INVALID);
    CONFIG_CASE(c_.window = 0, MD_E_INVALID);
    CONFIG_CASE(c_.quant_threshold = NAN, MD_E_INVALID);
    CONFIG_CASE(c_.head_dim = 64, MD_E_UNSUPPORTED);
    CONFIG_CASE(c_.window = 3, MD_E_UNSUPPORTED);            /* G W = 18 > 16 */
    CONFIG_CASE(c_.n_layers = 100, MD_E_UNSUPPORTED);        /* L Hq = 1200 rows */
    CONFIG_CASE(c_.page_size = 32, MD_E_UNSUPPORTED);
    CONFIG_CASE((c_.n_q_heads = 34, c_.n_kv_heads = 2, c_.n_layers = 2), MD_E_UNSUPPORTED);   /* G = 17 */
    CONFIG_CASE(c_.max_sessions = 1025, MD_E_UNSUPPORTED);
    CONFIG_CASE(c_.max_pages = 8193, MD_E_UNSUPPORTED);
    CONFIG_CASE((c_.page_size = 64, c_.n_phys_pages = 1 << 25), MD_E_UNSUPPORTED);   /* 2^31 slots */
}

static void view_cases(void) {
    const md_config c = good_config();
    md_cache_view v;
    float b[7 * 16], lam[7 * 16];
    md_region_params rp = {b, lam};
    md_handle h = NULL;

    EXPECT(md_init(NULL, &rp, &v, NULL, &h), MD_E_INVALID);
    v = good_view();
    EXPECT(md_init(&c, &rp, &v, NULL, NULL), MD_E_INVALID);
    EXPECT(md_init(&c, &rp, NULL, NULL, &h), MD_E_INVALID);
    EXPECT(md_init(&c, NULL, &v, NULL, &h), MD_E_INVALID);
    md_region_params rp_null = {NULL, lam};
    EXPECT(md_init(&c, &rp_null, &v, NULL, &h), MD_E_INVALID);
    md_region_params rp_odd = {(const float*)((const unsigned char*)b + 2), lam};
    EXPECT(md_init(&c, &rp_odd, &v, NULL, &h), MD_E_INVALID);

    v = good_view();
    v.k_pool = (uint16_t*)(arena + 8);              /* not 16-byte aligned */
    check_view(v, c, MD_E_INVALID, __LINE__);
    v = good_view();
    v.t_ref = (int32_t*)(arena + 3074);             /* not 4-byte aligned */
    check_view(v, c, MD_E_INVALID, __LINE__);
    v = good_view();
    v.free_count = NULL;
    check_view(v, c, MD_E_INVALID, __LINE__);

    md_config cq = good_config();
    cq.quant_threshold = 0.3f;
    v = good_view();                                 /* quantised tier without page formats */
    check_view(v, cq, MD_E_INVALID, __LINE__);

    md_config ca = good_config();
    ca.flags = MD_FLAG_REGION_ALIGNED;
    v = good_view();                                 /* region-aligned pages without n_live */
    check_view(v, ca, MD_E_INVALID, __LINE__);

    md_config co = good_config();
    co.offload_pages = 8;
    v = good_view();
    offload_view(&v);
    v.off_abar = NULL;                               /* offload tier with a missing array */
    check_view(v, co, MD_E_INVALID, __LINE__);
    v = good_view();
    offload_view(&v);
    v.host_keys = arena + 16384 + 4;                 /* host keys not 16-byte aligned */
    check_view(v, co, MD_E_INVALID, __LINE__);
}

static void handle_cases(void) {
    int32_t i32[8];
    int64_t i64[8];
    double ms = 0.0;
    float f32[4];
    uint64_t u64[4];
    uint8_t u8[4];
    EXPECT(md_observe_step(NULL, 1, f32, NULL, NULL, NULL), MD_E_INVALID);
    EXPECT(md_score_pages(NULL, NULL, NULL), MD_E_INVALID);
    EXPECT(md_select_evict(NULL, i32, i32, u8), MD_E_INVALID);
    EXPECT(md_compact(NULL, NULL, NULL), MD_E_INVALID);
    EXPECT(md_select_compact(NULL, i32, i32, u8), MD_E_INVALID);
    EXPECT(md_read_device_status(NULL, i32), MD_E_INVALID);
    EXPECT(md_profile_enable(NULL, 1u), MD_E_INVALID);
    EXPECT(md_profile_read(NULL, 0, &ms, i64), MD_E_INVALID);
    EXPECT(md_read_counters(NULL, i64), MD_E_INVALID);
    EXPECT(md_kernel_config(NULL, i32), MD_E_INVALID);
    EXPECT(md_calib_accumulate(NULL, f32, 8, 4, u64, u64, u64), MD_E_INVALID);
    EXPECT(md_destroy(NULL), MD_E_INVALID);
}

/* md_calib_fit on host arrays: an exact exponential law per region is
 * recovered (Eq. 6), a region with one usable bucket has no fit, and bad
 * arguments are refused. */
static void calib_cases(void) {
    enum { S = 2, R = 3, NB = 6 };
    uint64_t mass[S * R * NB], count[S * R * NB], age[S * R * NB];
    memset(mass, 0, sizeof(mass));
    memset(count, 0, sizeof(count));
    memset(age, 0, sizeof(age));
    const double lam_true[R] = {0.01, 0.05, 0.0};
    for (int s = 0; s < S; ++s)
        for (int r = 0; r < R; ++r)
            for (int b = 0; b < NB; ++b) {
                if (r == 2 && b > 0) continue;      /* region 2: a single bucket */
                const size_t k = ((size_t)s * R + r) * NB + b;
                const uint64_t n = 100;
                const double a = 8.0 * b + 4.0;     /* mean age of the bucket */
                const double m = 0.5 * exp(-lam_true[r] * a);
                count[k] = n;
                age[k] = (uint64_t)(a * n);
                mass[k] = (uint64_t)llround(m * n * 1099511627776.0);   /* 2^40 fixed point */
            }
    double lam[R], logc[R];
    EXPECT(md_calib_fit(mass, count, age, S, R, NB, lam, logc), MD_OK);
    for (int r = 0; r < 2; ++r)
        if (!(fabs(lam[r] - lam_true[r]) <= 1e-6 * fmax(lam_true[r], 1e-3)) || !(fabs(logc[r] - log(0.5)) <= 1e-6)) {
            fprintf(stderr, "calib region %d: lambda %.9g (want %.9g), log c %.9g\n", r, lam[r], lam_true[r], logc[r]);
            ++fails;
        }
    if (!isnan(lam[2]) || !isnan(logc[2])) {
        fprintf(stderr, "calib region 2: expected no fit, got %g\n", lam[2]);
        ++fails;
    }
    EXPECT(md_calib_fit(NULL, count, age, S, R, NB, lam, logc), MD_E_INVALID);
    EXPECT(md_calib_fit(mass, count, age, 0, R, NB, lam, logc), MD_E_INVALID);
    EXPECT(md_calib_fit(mass, count, age, S, R, 0, lam, logc), MD_E_INVALID);
    EXPECT(md_calib_fit(mass, count, age, S, R, NB, NULL, logc), MD_E_INVALID);
}

int main(void) {
    arena = (unsigned char*)aligned_alloc(256, 32768);
    if (arena == NULL) return 2;
    memset(arena, 0, 32768);
    if (md_abi_version() != MD_ABI_VERSION) {
        fprintf(stderr, "ABI %d, header %d\n", md_abi_version(), MD_ABI_VERSION);
        ++fails;
    }
    for (int s = -8; s <= 2; ++s) {
        const char* t = md_status_str((md_status)s);
        if (t == NULL || t[0] == '\0') {
            fprintf(stderr, "md_status_str(%d) empty\n", s);
            ++fails;
        }
    }
    config_cases();
    view_cases();
    handle_cases();
    calib_cases();
    free(arena);
    if (fails == 0) printf("host ABI checks passed under the sanitizers\n");
    return fails == 0 ? 0 : 1;
}
