/* A C99 program that uses the host-only calls of librhymeflow.so through
   include/rhymeflow.h (no GPU needed): it shows that the header is plain C
   and prints results that tests/test_c_header.py checks against the oracle. */
#include <stdio.h>
#include <string.h>

#include "rhymeflow.h"

int main(void) {
    int32_t ids[RF_MAX_FRAMES], n = 0;
    uint8_t mask[RF_MAX_FRAMES];
    const int32_t given[4] = {12, 4, 4, 20};
    int i;

    printf("abi %d\n", rf_abi_version());
    if (rf_select_keyframes(given, 4, 21, 0u, ids, &n, mask) != RF_OK) return 1;
    printf("select");
    for (i = 0; i < n; ++i) printf(" %d", ids[i]);
    printf("\n");
    if (rf_keyframes_uniform(21, 6, ids, &n) != RF_OK) return 1;
    printf("uniform");
    for (i = 0; i < n; ++i) printf(" %d", ids[i]);
    printf("\n");

    {   /* Alg. 1 on a block-structured similarity matrix: scenes of 4 frames */
        double sim[16 * 16];
        int r, c;
        for (r = 0; r < 16; ++r)
            for (c = 0; c < 16; ++c) sim[r * 16 + c] = (r / 4 == c / 4) ? 0.9 : 0.1;
        if (rf_select_keyframes_adaptive(sim, 16, 0.5, 8, 0.05, 1.0, 1.0, 0u, ids, &n, NULL) != RF_OK) return 1;
        printf("adaptive");
        for (i = 0; i < n; ++i) printf(" %d", ids[i]);
        printf("\n");
    }

    {   /* Eq. 2 / Alg. 2 */
        rf_step_plan plan[50];
        int32_t nr = 0, ns = 0;
        if (rf_async_schedule(50, 8, 25, 2, 3, plan, &nr, &ns) != RF_OK) return 1;
        printf("schedule %d %d", nr, ns);
        for (i = 0; i < 50; ++i)
            if (plan[i].phase == RF_STEP_RHYTHMIC) printf(" %d", plan[i].t);
        printf("\n");
    }

    {   /* the rolling cache's bookkeeping (App. B.2) without device copies */
        rf_rolling_cache cache;
        const int32_t frames[3] = {1, 2, 4};
        double a = 0.0;
        memset(&cache, 0, sizeof cache);
        if (rf_cache_init(&cache, NULL, NULL, frames, 3, 5, 16, 64, RF_BF16, 24.0, NULL) != RF_OK) return 1;
        if (rf_cache_shift_store(&cache, NULL, NULL, NULL, 0, 21.0, NULL) != RF_OK) return 1;
        if (rf_cache_alpha(&cache, 2, 23.0, &a) != RF_OK) return 1;
        printf("cache %d %d %d %d %.17g\n", cache.before_slot[2], cache.after_slot[2], cache.before_slot[4],
               cache.after_slot[4], a);
    }

    {   /* workspace and plan of the split-key tail at 33 x 45 x 80, 24 heads, on 256 compute units */
        int64_t bytes = 0;
        rf_attention_split plan;
        if (rf_attention_workspace(8, 33, 33, 45, 80, 24, 128, RF_BF16, 256, &bytes) != RF_OK) return 1;
        if (rf_attention_plan(8, 33, 33, 45, 80, 24, 128, RF_BF16, 256, &plan) != RF_OK) return 1;
        printf("workspace %lld\n", (long long)bytes);
        printf("plan %lld %lld %lld %d %d %lld %d\n", (long long)plan.tiles, (long long)plan.whole_tiles,
               (long long)plan.tail_tiles, plan.parts, plan.key_tiles_per_part, (long long)plan.workspace_bytes,
               plan.compute_units);
    }

    /* an error: described, nothing written */
    n = -7;
    if (rf_keyframes_uniform(21, 30, ids, &n) != RF_ERR_RANGE) return 1;
    printf("error %s n=%d msg=%s\n", rf_status_string(RF_ERR_RANGE), n, rf_last_error());
    return 0;
}
