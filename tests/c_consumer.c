/* A plain C99 consumer of the C ABI (include/infs.h), built and run by
 * tests/test_c_consumer.py on a host without a GPU: a dry-run context runs the
 * group decode loop of one prompt under a host scheduler, with the state
 * machine's error paths, and the FPTAS grouping.  Prints key = value lines. */
#include <stdio.h>
#include <string.h>

#include "infs.h"

#define G 10
#define M 4
#define LAYERS 2

static int fail(const char* what, infs_status st, const infs_ctx* ctx) {
    printf("error %s: status %d: %s\n", what, (int)st, infs_last_error(ctx));
    return 1;
}

int main(int argc, char** argv) {
    static const int32_t lengths[G] = {5, 17, 3, 9, 12, 1, 30, 8, 8, 2};
    static const double pred[G] = {6.0, 15.5, 2.5, 11.0, 12.0, 1.5, 28.0, 7.0, 9.0, 2.0};
    int policy = INFS_SJF;
    infs_config cfg;
    infs_ctx* ctx = NULL;
    infs_sched* sched = NULL;
    infs_stats stats;
    infs_kernel_info info;
    int32_t slot_sample[M], slot_len[M];
    int32_t group[G], pos[G];
    int64_t steps = 0;
    int done = 0, s, l, i;
    infs_status st;

    if (argc > 1) policy = argv[1][0] - '0';
    if (infs_abi_version() != INFS_ABI_VERSION) {
        printf("error abi version %d\n", (int)infs_abi_version());
        return 1;
    }
    memset(&cfg, 0, sizeof cfg);
    cfg.num_layers = LAYERS;
    cfg.num_q_heads = 4;
    cfg.num_kv_heads = 2;
    cfg.head_dim = 64;
    cfg.num_prompts = 1;
    cfg.slots_per_prompt = M;
    cfg.samples_per_prompt = G;
    cfg.max_prompt_len = 32;
    cfg.max_suffix_len = 64;
    cfg.dtype = INFS_F32;
    cfg.flags = INFS_FLAG_DRY_RUN;
    st = infs_create(&cfg, NULL, &ctx);
    if (st != INFS_OK) return fail("create", st, NULL);
    st = infs_get_kernel_info(ctx, &info);
    if (st != INFS_OK) return fail("kernel_info", st, ctx);
    printf("kernel = bf16 %d head_dim %d hpk %d mfma %d rows %d\n", (int)info.bf16, (int)info.head_dim,
           (int)info.hpk, (int)info.mfma, (int)info.prefix_rows);

    /* Layer 0's prefix now; layer 1's after the first refills, to show that decoding a layer whose
       prefix is not in place (with live slots) is a state error that leaves the context as it was. */
    st = infs_prefill_shared(ctx, 0, 0, 32, NULL, NULL);
    if (st != INFS_OK) return fail("prefill", st, ctx);
    st = infs_sched_create(G, M, policy, pred, &sched);
    if (st != INFS_OK) return fail("sched_create", st, NULL);

    for (s = 0; s < M; ++s) slot_sample[s] = -1;
    for (;;) {
        for (s = 0; s < M; ++s) {
            if (slot_sample[s] >= 0) continue;
            {
                int64_t id = -1;
                st = infs_sched_next(sched, s, &id);
                if (st != INFS_OK) return fail("sched_next", st, NULL);
                if (id < 0) continue;
                st = infs_refill_slot(ctx, s, 0, id);
                if (st != INFS_OK) return fail("refill", st, ctx);
                slot_sample[s] = (int32_t)id;
                slot_len[s] = 0;
            }
        }
        if (done == G) break;
        if (steps == 0) {
            st = infs_refill_slot(ctx, 0, 0, 0);
            printf("refill_live_slot = %d (%s)\n", (int)st, infs_last_error(ctx));
            st = infs_decode_step(ctx, 1, NULL, NULL, NULL, NULL);
            printf("decode_before_prefill = %d (%s)\n", (int)st, infs_last_error(ctx));
            st = infs_prefill_shared(ctx, 0, 1, 32, NULL, NULL);
            if (st != INFS_OK) return fail("prefill", st, ctx);
        }
        for (l = 0; l < LAYERS; ++l) {
            st = infs_decode_step(ctx, l, NULL, NULL, NULL, NULL);
            if (st != INFS_OK) return fail("decode", st, ctx);
        }
        if (steps == 0) printf("second_decode_same_layer = %d\n", (int)infs_decode_step(ctx, 0, NULL, NULL, NULL, NULL));
        st = infs_end_step(ctx);
        if (st != INFS_OK) return fail("end_step", st, ctx);
        ++steps;
        for (s = 0; s < M; ++s) {
            if (slot_sample[s] < 0) continue;
            if (++slot_len[s] == lengths[slot_sample[s]]) {
                st = infs_retire_slot(ctx, s);
                if (st != INFS_OK) return fail("retire", st, ctx);
                st = infs_sched_done(sched, s);
                if (st != INFS_OK) return fail("sched_done", st, NULL);
                slot_sample[s] = -1;
                ++done;
            }
        }
    }
    st = infs_retire_slot(ctx, 0);
    printf("retire_empty_slot = %d\n", (int)st);
    st = infs_get_stats(ctx, &stats);
    if (st != INFS_OK) return fail("stats", st, ctx);
    printf("steps = %lld\n", (long long)steps);
    printf("stats_steps = %lld\n", (long long)stats.steps);
    printf("launches = %lld\n", (long long)stats.launches);
    printf("tokens = %lld\n", (long long)stats.tokens);
    infs_sched_destroy(sched);
    infs_destroy(ctx);

    st = infs_fptas_assign(G, M, pred, INFS_FPTAS_EPSILON, group, pos);
    if (st != INFS_OK) return fail("fptas", st, NULL);
    printf("fptas_group =");
    for (i = 0; i < G; ++i) printf(" %d", (int)group[i]);
    printf("\nfptas_pos =");
    for (i = 0; i < G; ++i) printf(" %d", (int)pos[i]);
    printf("\n");
    return 0;
}
