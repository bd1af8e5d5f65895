/*
 * The host side of the C ABI under AddressSanitizer and UndefinedBehaviorSanitizer:
 * every entry point driven through its argument checks (NULL pointers, sizes
 * that are zero, negative or whose byte counts overflow, id lists out of range,
 * unsorted or too long, misaligned or overlapping buffers, corrupted cache
 * structs, non-finite times), plus the host-only calls that succeed, writing
 * into outputs allocated to their exact documented size so that any write past
 * them is caught. No call reaches a kernel launch: device pointers are
 * fabricated addresses that the checks reject, and nothing is dereferenced.
 * Prints "ok <number of checks>" and exits 0, or names the first failing check.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "rhymeflow.h"

static int checks = 0;

#define EXPECT(call, want)                                                                      \
    do {                                                                                        \
        const int got_ = (call);                                                                \
        ++checks;                                                                               \
        if (got_ != (want)) {                                                                   \
            printf("FAIL line %d: %s returned %d, expected %d (%s)\n", __LINE__, #call, got_,   \
                   (int)(want), rf_last_error());                                               \
            return 1;                                                                           \
        }                                                                                       \
    } while (0)

/* fabricated, 256-byte aligned device addresses, far apart (never dereferenced) */
#define DEV(i) ((void *)(uintptr_t)(0x100000000000ull + (uint64_t)(i) * 0x10000000000ull))

int main(void) {
    const int32_t T = 9;
    int32_t *ids = (int32_t *)malloc(sizeof(int32_t) * T);    /* capacity T, exactly */
    uint8_t *mask = (uint8_t *)malloc((size_t)T);
    int32_t n = -1;

    /* --- keyframe sets --- */
    {
        const int32_t in[4] = {4, 8, 4, 2};
        EXPECT(rf_select_keyframes(in, 4, T, 0, ids, &n, mask), RF_OK);
        if (n != 4 || ids[0] != 0 || ids[3] != 8 || mask[8] != 1 || mask[1] != 0) return printf("select\n"), 1;
        int32_t all[9] = {8, 7, 6, 5, 4, 3, 2, 1, 0};
        EXPECT(rf_select_keyframes(all, 9, T, 0, ids, &n, mask), RF_OK);
        EXPECT(rf_select_keyframes(in, 4, T, 0, NULL, &n, mask), RF_ERR_INVALID_ARG);
        EXPECT(rf_select_keyframes(in, -1, T, 0, ids, &n, mask), RF_ERR_INVALID_ARG);
        EXPECT(rf_select_keyframes(NULL, 2, T, 0, ids, &n, mask), RF_ERR_INVALID_ARG);
        EXPECT(rf_select_keyframes(in, 4, 0, 0, ids, &n, mask), RF_ERR_RANGE);
        EXPECT(rf_select_keyframes(in, 4, RF_MAX_FRAMES + 1, 0, ids, &n, mask), RF_ERR_RANGE);
        EXPECT(rf_select_keyframes(in, 4, 4, 0, ids, &n, mask), RF_ERR_RANGE);        /* id 8 >= 4 */
        const int32_t neg[1] = {-1};
        EXPECT(rf_select_keyframes(neg, 1, T, 0, ids, &n, mask), RF_ERR_RANGE);
        EXPECT(rf_select_keyframes(NULL, 0, T, RF_SEL_NO_FORCE_FIRST, ids, &n, mask), RF_ERR_INVALID_ARG);
        EXPECT(rf_select_keyframes(in, 4, T, 0x80u, ids, &n, mask), RF_ERR_INVALID_ARG);
        EXPECT(rf_keyframes_stride(T, 1, ids, &n), RF_OK);
        EXPECT(rf_keyframes_stride(T, 0, ids, &n), RF_ERR_INVALID_ARG);
        EXPECT(rf_keyframes_stride(-3, 2, ids, &n), RF_ERR_RANGE);
        EXPECT(rf_keyframes_stride(T, 2, NULL, &n), RF_ERR_INVALID_ARG);
        EXPECT(rf_keyframes_uniform(T, T, ids, &n), RF_OK);
        EXPECT(rf_keyframes_uniform(T, 1, ids, &n), RF_OK);
        EXPECT(rf_keyframes_uniform(T, T + 1, ids, &n), RF_ERR_RANGE);
        EXPECT(rf_keyframes_uniform(T, 0, ids, &n), RF_ERR_RANGE);
        EXPECT(rf_keyframes_uniform(T, 3, ids, NULL), RF_ERR_INVALID_ARG);
    }

    /* --- projection --- */
    {
        const double ts[3] = {24.0, 21.0, 23.0};
        const double bad[3] = {24.0, NAN, 23.0};
        uint8_t m5[5] = {1, 0, 1, 0, 1};
        EXPECT(rf_project_latents(NULL, DEV(1), ts, m5, 1, 4, 5, 8, 8, RF_F32, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_project_latents(DEV(0), DEV(1), NULL, m5, 1, 4, 5, 8, 8, RF_F32, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_project_latents(DEV(0), DEV(1), ts, NULL, 1, 4, 5, 8, 8, RF_F32, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_project_latents(DEV(0), DEV(1), ts, m5, 0, 4, 5, 8, 8, RF_F32, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_project_latents(DEV(0), DEV(1), ts, m5, 1, 4, 300, 8, 8, RF_F32, NULL), RF_ERR_RANGE);
        EXPECT(rf_project_latents(DEV(0), DEV(1), ts, m5, 1, 4, 5, 8, 8, 7, NULL), RF_ERR_UNSUPPORTED);
        EXPECT(rf_project_latents(DEV(0), DEV(1), ts, m5, 2147483647, 2147483647, 5, 8, 8, RF_F32, NULL),
               RF_ERR_RANGE);
        EXPECT(rf_project_latents(DEV(0), DEV(1), bad, m5, 1, 4, 5, 8, 8, RF_F32, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_project_latents((char *)DEV(0) + 4, DEV(1), ts, m5, 1, 4, 5, 8, 8, RF_F32, NULL),
               RF_ERR_UNSUPPORTED);
        EXPECT(rf_project_latents(DEV(0), (char *)DEV(0) + 64, ts, m5, 1, 4, 5, 8, 8, RF_F32, NULL),
               RF_ERR_INVALID_ARG);                                                   /* overlap */
    }

    /* --- attention family --- */
    {
        const int32_t kf[3] = {0, 4, 8};
        const int32_t dup[3] = {0, 4, 4};
        const int32_t far[3] = {0, 4, 9};
        int32_t *many = (int32_t *)malloc(sizeof(int32_t) * (RF_MAX_FRAMES + 1));
        for (int i = 0; i <= RF_MAX_FRAMES; ++i) many[i] = i;
        EXPECT(rf_keyframe_attention(NULL, DEV(1), DEV(2), DEV(3), kf, 3, T, 8, 8, 2, 128, RF_BF16, NULL),
               RF_ERR_INVALID_ARG);
        EXPECT(rf_keyframe_attention(DEV(0), DEV(1), DEV(2), DEV(3), NULL, 3, T, 8, 8, 2, 128, RF_BF16, NULL),
               RF_ERR_INVALID_ARG);
        EXPECT(rf_keyframe_attention(DEV(0), DEV(1), DEV(2), DEV(3), kf, 0, T, 8, 8, 2, 128, RF_BF16, NULL),
               RF_ERR_INVALID_ARG);
        EXPECT(rf_keyframe_attention(DEV(0), DEV(1), DEV(2), DEV(3), dup, 3, T, 8, 8, 2, 128, RF_BF16, NULL),
               RF_ERR_INVALID_ARG);
        EXPECT(rf_keyframe_attention(DEV(0), DEV(1), DEV(2), DEV(3), far, 3, T, 8, 8, 2, 128, RF_BF16, NULL),
               RF_ERR_RANGE);
        EXPECT(rf_keyframe_attention(DEV(0), DEV(1), DEV(2), DEV(3), many, RF_MAX_FRAMES + 1, RF_MAX_FRAMES + 1, 1,
                                     1, 2, 128, RF_BF16, NULL), RF_ERR_RANGE);
        EXPECT(rf_keyframe_attention(DEV(0), DEV(1), DEV(2), DEV(3), kf, 3, T, 8, 8, 2, 96, RF_BF16, NULL),
               RF_ERR_UNSUPPORTED);
        EXPECT(rf_keyframe_attention(DEV(0), DEV(1), DEV(2), DEV(3), kf, 3, T, 8, 8, 2, 128, 5, NULL),
               RF_ERR_UNSUPPORTED);
        EXPECT(rf_keyframe_attention(DEV(0), DEV(1), DEV(2), DEV(3), kf, 3, T, 2147483647, 2147483647, 8, 128,
                                     RF_BF16, NULL), RF_ERR_RANGE);
        EXPECT(rf_keyframe_attention(DEV(0), (char *)DEV(1) + 8, DEV(2), DEV(3), kf, 3, T, 8, 8, 2, 128, RF_BF16,
                                     NULL), RF_ERR_UNSUPPORTED);
        EXPECT(rf_keyframe_attention(DEV(0), DEV(1), DEV(2), (char *)DEV(2) + 256, kf, 3, T, 8, 8, 2, 128, RF_BF16,
                                     NULL), RF_ERR_INVALID_ARG);                      /* out inside v */
        EXPECT(rf_keyframe_attention_ws(DEV(0), DEV(1), DEV(2), DEV(3), kf, 3, T, 8, 8, 2, 128, RF_BF16, NULL, 0,
                                        NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_keyframe_attention_ws(DEV(0), DEV(1), DEV(2), DEV(3), kf, 3, T, 8, 8, 2, 128, RF_BF16, DEV(4),
                                        -5, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_keyframe_attention_ws(DEV(0), DEV(1), DEV(2), DEV(3), kf, 3, T, 8, 8, 2, 128, RF_BF16,
                                        (char *)DEV(4) + 8, 1 << 20, NULL), RF_ERR_UNSUPPORTED);
        EXPECT(rf_keyframe_attention_ws(DEV(0), DEV(1), DEV(2), DEV(3), kf, 3, T, 8, 8, 2, 128, RF_BF16,
                                        (char *)DEV(0) + 512, 1 << 20, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_keyframe_attention_noalloc(DEV(0), DEV(1), DEV(2), DEV(3), dup, 3, T, 8, 8, 2, 128, RF_BF16,
                                             NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_keyframe_attention_noalloc(DEV(0), DEV(1), DEV(2), NULL, kf, 3, T, 8, 8, 2, 128, RF_BF16,
                                             NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_frame_attention(DEV(0), DEV(1), DEV(2), DEV(3), kf, 3, NULL, 2, T, 8, 8, 2, 64, RF_BF16, NULL,
                                  0, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_frame_attention(DEV(0), DEV(1), DEV(2), DEV(3), kf, 3, dup, 3, T, 8, 8, 2, 64, RF_BF16, NULL,
                                  0, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_frame_attention(DEV(0), DEV(1), DEV(2), DEV(3), kf, 3, many, RF_MAX_FRAMES + 1, T, 8, 8, 2, 64,
                                  RF_BF16, NULL, 0, NULL), RF_ERR_RANGE);
        int64_t bytes = -1;
        rf_attention_split *plan = (rf_attention_split *)malloc(sizeof *plan);
        EXPECT(rf_attention_workspace(8, 33, 33, 45, 80, 24, 128, RF_BF16, 256, &bytes), RF_OK);
        if (bytes != 152LL * 5 * 256 * 520) return printf("workspace %lld\n", (long long)bytes), 1;
        EXPECT(rf_attention_plan(8, 33, 33, 45, 80, 24, 128, RF_BF16, 80, plan), RF_OK);
        EXPECT(rf_attention_plan(8, 33, 33, 45, 80, 24, 128, RF_F32, 1, plan), RF_OK);
        EXPECT(rf_attention_plan(8, 33, 33, 45, 80, 24, 128, RF_BF16, RF_MAX_COMPUTE_UNITS + 1, plan), RF_ERR_RANGE);
        EXPECT(rf_attention_plan(8, 33, 33, 45, 80, 24, 128, RF_BF16, -2, plan), RF_ERR_RANGE);
        EXPECT(rf_attention_plan(8, 33, 33, 45, 80, 24, 128, RF_BF16, 256, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_attention_workspace(0, 33, 33, 45, 80, 24, 128, RF_BF16, 256, &bytes), RF_ERR_INVALID_ARG);
        EXPECT(rf_attention_workspace(9, 8, 8, 45, 80, 24, 128, RF_BF16, 256, &bytes), RF_ERR_RANGE);
        EXPECT(rf_attention_workspace(2, 4, 4, 2147483647, 2147483647, 8, 128, RF_BF16, 256, &bytes), RF_ERR_RANGE);
        free(plan);
        free(many);
    }

    /* --- gather / scatter --- */
    {
        const int32_t fr[2] = {1, 3};
        const int32_t rev[2] = {3, 1};
        EXPECT(rf_gather_frames(NULL, DEV(1), fr, 2, 4, 16, 256, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_gather_frames(DEV(0), DEV(1), rev, 2, 4, 16, 256, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_gather_frames(DEV(0), DEV(1), fr, 2, 4, 16, 24, NULL), RF_ERR_UNSUPPORTED);
        EXPECT(rf_gather_frames(DEV(0), DEV(1), fr, 2, 4, 0, 256, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_gather_frames(DEV(0), DEV(1), fr, 2, 4, 1LL << 40, 1LL << 32, NULL), RF_ERR_RANGE);
        EXPECT(rf_scatter_frames(DEV(0), (char *)DEV(0) + 4096, fr, 2, 4, 16, 256, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_scatter_frames(DEV(0), DEV(1), fr, 2, 3, 16, 256, NULL), RF_ERR_RANGE);   /* frame 3 >= T */
    }

    /* --- frame similarity and Alg. 1's scan --- */
    {
        int64_t bytes = -1;
        EXPECT(rf_frame_similarity_workspace(1, 16, 33, 90, 160, &bytes), RF_OK);
        EXPECT(rf_frame_similarity_workspace(1, 16, 0, 90, 160, &bytes), RF_ERR_INVALID_ARG);
        EXPECT(rf_frame_similarity_workspace(1, 16, 300, 90, 160, &bytes), RF_ERR_RANGE);
        EXPECT(rf_frame_similarity_workspace(1, 16, 33, 90, 160, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_frame_similarity(DEV(0), (double *)DEV(1), NULL, 1 << 20, 1, 16, 33, 90, 160, RF_F32, NULL),
               RF_ERR_INVALID_ARG);
        EXPECT(rf_frame_similarity(DEV(0), (double *)DEV(1), DEV(2), 16, 1, 16, 33, 90, 160, RF_F32, NULL),
               RF_ERR_INVALID_ARG);
        EXPECT(rf_frame_similarity(DEV(0), (double *)DEV(1), DEV(2), 1LL << 40, 1, 16, 33, 90, 160, 9, NULL),
               RF_ERR_UNSUPPORTED);
        double *sim = (double *)malloc(sizeof(double) * T * T);
        for (int i = 0; i < T * T; ++i) sim[i] = (i / T) / 3 == (i % T) / 3 ? 0.9 : 0.1;
        EXPECT(rf_select_keyframes_adaptive(sim, T, 0.5, 4, 0.05, 1.0, 1.0, 0, ids, &n, mask), RF_OK);
        EXPECT(rf_select_keyframes_adaptive(sim, T, 0.5, T, 0.05, 1.0, 1.0, RF_SEL_INTENT_SIGN, ids, &n, mask),
               RF_OK);
        EXPECT(rf_select_keyframes_adaptive(sim, T, NAN, 4, 0.05, 1.0, 1.0, 0, ids, &n, mask), RF_ERR_INVALID_ARG);
        EXPECT(rf_select_keyframes_adaptive(sim, T, 0.5, T + 1, 0.05, 1.0, 1.0, 0, ids, &n, mask), RF_ERR_RANGE);
        EXPECT(rf_select_keyframes_adaptive(sim, T, 0.5, 4, 0.05, 1.0, 1.0, 0x4u, ids, &n, mask),
               RF_ERR_INVALID_ARG);
        EXPECT(rf_select_keyframes_adaptive(NULL, T, 0.5, 4, 0.05, 1.0, 1.0, 0, ids, &n, mask), RF_ERR_INVALID_ARG);
        free(sim);
    }

    /* --- rolling cache bookkeeping --- */
    {
        rf_rolling_cache *c = (rf_rolling_cache *)malloc(sizeof *c);
        const int32_t nk[3] = {1, 2, 5};
        int64_t bytes = -1;
        double a = -1.0;
        EXPECT(rf_cache_store_bytes(3, 16, 64, RF_BF16, &bytes), RF_OK);
        EXPECT(rf_cache_store_bytes(0, 16, 64, RF_BF16, &bytes), RF_ERR_INVALID_ARG);
        EXPECT(rf_cache_store_bytes(RF_MAX_FRAMES + 1, 16, 64, RF_BF16, &bytes), RF_ERR_RANGE);
        EXPECT(rf_cache_store_bytes(3, 1LL << 50, 1 << 20, RF_F32, &bytes), RF_ERR_RANGE);
        memset(c, 0, sizeof *c);
        EXPECT(rf_cache_alpha(c, 1, 20.0, &a), RF_ERR_INVALID_ARG);                    /* never initialised */
        EXPECT(rf_cache_init(c, NULL, NULL, nk, 3, T, 16, 64, RF_BF16, 24.0, NULL), RF_OK);
        EXPECT(rf_cache_init(c, NULL, NULL, nk, 3, T, 16, 64, RF_BF16, INFINITY, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_cache_init(c, NULL, NULL, nk, 3, T, 16, 4, RF_BF16, 24.0, NULL), RF_ERR_UNSUPPORTED);
        EXPECT(rf_cache_init(c, NULL, DEV(1), nk, 3, T, 16, 64, RF_BF16, 24.0, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_cache_shift_store(c, NULL, NULL, NULL, 0, 21.0, NULL), RF_OK);
        EXPECT(rf_cache_shift_store(c, NULL, NULL, NULL, 0, 22.0, NULL), RF_ERR_INVALID_ARG);   /* not below */
        EXPECT(rf_cache_alpha(c, 2, 23.0, &a), RF_OK);
        if (!(a > 0.3 && a < 0.34)) return printf("alpha %g\n", a), 1;
        EXPECT(rf_cache_alpha(c, 3, 23.0, &a), RF_ERR_INVALID_ARG);                    /* not cached */
        EXPECT(rf_cache_alpha(c, T, 23.0, &a), RF_ERR_RANGE);
        EXPECT(rf_cache_alpha(c, 2, NAN, &a), RF_ERR_INVALID_ARG);
        const int32_t sub[1] = {5};
        const int32_t notc[1] = {4};
        EXPECT(rf_cache_shift_store(c, NULL, NULL, sub, 1, 18.0, NULL), RF_OK);
        EXPECT(rf_cache_shift_store(c, NULL, NULL, notc, 1, 15.0, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_cache_project_kv(c, NULL, DEV(1), DEV(2), NULL, 0, 20.0, NULL), RF_ERR_INVALID_ARG);
        EXPECT(rf_cache_project_kv(c, DEV(0), DEV(1), DEV(1), NULL, 0, 20.0, NULL), RF_ERR_INVALID_ARG);
        rf_rolling_cache *bad = (rf_rolling_cache *)malloc(sizeof *bad);
        memcpy(bad, c, sizeof *bad);
        bad->after_slot[2] = 200;                                                      /* out of its pair */
        EXPECT(rf_cache_alpha(bad, 2, 23.0, &a), RF_ERR_INVALID_ARG);
        memcpy(bad, c, sizeof *bad);
        bad->t_after[1] = NAN;
        EXPECT(rf_cache_alpha(bad, 1, 23.0, &a), RF_ERR_INVALID_ARG);
        memcpy(bad, c, sizeof *bad);
        bad->T = 1000;
        EXPECT(rf_cache_alpha(bad, 1, 23.0, &a), RF_ERR_INVALID_ARG);
        memcpy(bad, c, sizeof *bad);
        bad->rows_per_frame = 1LL << 62;
        EXPECT(rf_cache_alpha(bad, 1, 23.0, &a), RF_ERR_INVALID_ARG);
        free(bad);
        free(c);
    }

    /* --- schedule --- */
    {
        rf_step_plan *plan = (rf_step_plan *)malloc(sizeof(rf_step_plan) * 50);
        int32_t nr = -1, ns = -1;
        EXPECT(rf_async_schedule(50, 8, 25, 2, 3, plan, &nr, &ns), RF_OK);
        if (nr != 17 || ns != 25) return printf("schedule %d %d\n", nr, ns), 1;
        EXPECT(rf_async_schedule(50, 51, 25, 2, 3, plan, &nr, &ns), RF_ERR_RANGE);
        EXPECT(rf_async_schedule(50, 8, 25, 0, 3, plan, &nr, &ns), RF_ERR_INVALID_ARG);
        EXPECT(rf_async_schedule(0, 0, 0, 1, 1, plan, &nr, &ns), RF_ERR_RANGE);
        EXPECT(rf_async_schedule(50, 8, 25, 2, 3, NULL, &nr, &ns), RF_ERR_INVALID_ARG);
        free(plan);
    }

    /* --- probes --- */
    EXPECT(rf_probe_mfma_bf16(NULL, 1, 1, (float *)DEV(1), NULL), RF_ERR_INVALID_ARG);
    EXPECT(rf_probe_mfma_bf16(DEV(0), 0, 1, (float *)DEV(1), NULL), RF_ERR_RANGE);
    EXPECT(rf_probe_hbm_read(DEV(0), 17, 1, (uint32_t *)DEV(1), NULL), RF_ERR_INVALID_ARG);
    EXPECT(rf_probe_hbm_read(DEV(0), 4096, 0, (uint32_t *)DEV(1), NULL), RF_ERR_RANGE);
    EXPECT(rf_probe_lds_read(1, 1, 16, NULL, NULL, NULL), RF_ERR_INVALID_ARG);
    EXPECT(rf_probe_lds_read(1, 1, 12, (uint32_t *)DEV(1), NULL, NULL), RF_ERR_INVALID_ARG);
    EXPECT(rf_probe_lds_read(1, 0, 8, (uint32_t *)DEV(1), NULL, NULL), RF_ERR_RANGE);
    EXPECT(rf_probe_lds_read(1, 1, 8, (uint32_t *)DEV(1), (uint64_t *)((char *)DEV(0) + 4), NULL),
           RF_ERR_UNSUPPORTED);

    /* every status has a name; an unknown one too */
    for (int s = -6; s <= 1; ++s)
        if (!rf_status_string(s) || !rf_status_string(s)[0]) return printf("status string %d\n", s), 1;
    if (rf_abi_version() != RF_ABI_VERSION) return printf("abi version\n"), 1;

    free(ids);
    free(mask);
    printf("ok %d\n", checks);
    return 0;
}
