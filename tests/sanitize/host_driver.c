/*
 * Address/undefined-behaviour sanitizer run of libpdec's host logic: the
 * dims checks, the planner, workspace sizing, the length contract check on
 * host arrays, the path and timer settings and the argument checks of every
 * launching entry point.  tests/test_sanitizers.py links this driver with the
 * library's sources compiled for the host only (no device code), so nothing
 * here may reach a kernel launch: every launching call gets an argument that
 * the library refuses first.  Exit status 0: no error.
 */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "pdec.h"

#define CHECK(c)                                                          \
    do {                                                                  \
        if (!(c)) {                                                       \
            fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            return 1;                                                     \
        }                                                                 \
    } while (0)

static pdec_dims dims(int E, int hq, int hkv, int d, int cap, int L, int dtype)
{
    pdec_dims x;
    memset(&x, 0, sizeof(x));
    x.num_events = E;
    x.num_q_heads = hq;
    x.num_kv_heads = hkv;
    x.head_dim = d;
    x.event_cap = cap;
    x.max_prefix_len = L;
    x.dtype = dtype;
    return x;
}

/* Fake, suitably aligned, never-dereferenced device addresses: every call
 * that receives them is refused before it touches device memory. */
#define FAKE(n) ((void*)(uintptr_t)(0x100000u * (n)))

static int planner_sweep(void)
{
    const int Es[] = {1, 3, 7, 16, 32, 100, 2048, 2049};
    const int Ds[] = {64, 128, 96};
    const int Ls[] = {0, 1, 63, 64, 65, 32768, 1 << 20};
    const int caps[] = {1, 64, 129, 4096};
    for (unsigned a = 0; a < sizeof(Es) / sizeof(Es[0]); ++a)
        for (unsigned b = 0; b < sizeof(Ds) / sizeof(Ds[0]); ++b)
            for (unsigned c = 0; c < sizeof(Ls) / sizeof(Ls[0]); ++c)
                for (unsigned e = 0; e < sizeof(caps) / sizeof(caps[0]); ++e)
                    for (int dt = 0; dt < 2; ++dt)
                        for (int qps = 0; qps < 3; qps += 2) {
                            pdec_dims x = dims(Es[a], 28, 4, Ds[b], caps[e], Ls[c], dt);
                            x.queries_per_stream = qps;
                            for (int v = 1; v <= 3; v += 2) {
                                const size_t ws = pdec_workspace_size(&x, v);
                                int32_t path = -7, chunk = -7;
                                const int rc = pdec_query_plan(&x, v, &path, &chunk);
                                pdec_plan_info info;
                                const int rc2 = pdec_describe_plan(&x, v, &info);
                                CHECK(rc == rc2);
                                CHECK((rc == PDEC_OK) == (ws > 0));
                                if (rc == PDEC_OK) {
                                    CHECK(path == 1 || path == 2);
                                    CHECK(chunk > 0 && chunk % 64 == 0);
                                    CHECK(info.max_chunks >= 1 && info.work_items >= 1);
                                    CHECK(info.chunk_keys == chunk);
                                }
                            }
                        }
    /* each field out of range */
    pdec_dims bad[12];
    for (int i = 0; i < 12; ++i) bad[i] = dims(32, 28, 4, 128, 129, 32768, PDEC_DTYPE_BF16);
    bad[0].num_events = 0;
    bad[1].num_q_heads = 0;
    bad[2].num_kv_heads = 3;
    bad[3].head_dim = 0;
    bad[4].event_cap = 0;
    bad[5].max_prefix_len = -1;
    bad[6].dtype = 7;
    bad[7].softmax_scale = 1.0f / 0.0f;
    bad[8].plan_mask = 2;
    bad[9].plan_tokens_per_stream = -1;
    bad[10].queries_per_stream = -2;
    bad[11].cross_causal = 1;
    for (int i = 0; i < 12; ++i) {
        int32_t path, chunk;
        CHECK(pdec_workspace_size(&bad[i], 1) == 0);
        CHECK(pdec_query_plan(&bad[i], 1, &path, &chunk) != PDEC_OK);
    }
    CHECK(pdec_workspace_size(NULL, 1) == 0);
    pdec_dims ok = dims(32, 28, 4, 128, 129, 32768, PDEC_DTYPE_BF16);
    CHECK(pdec_workspace_size(&ok, 0) == 0);
    return 0;
}

static int lengths(void)
{
    pdec_dims x = dims(4, 28, 4, 128, 10, 100, PDEC_DTYPE_BF16);
    x.max_events_per_video = 3;
    x.prefix_tokens = 150;
    const int32_t ev_ok[4] = {0, 10, 3, 1}, ev_neg[4] = {0, -1, 3, 1}, ev_big[4] = {0, 11, 3, 1};
    const int32_t pl_ok[1] = {100}, pl_big[1] = {101}, pl_neg[1] = {-1};
    CHECK(pdec_check_lengths(&x, 1, ev_ok, pl_ok, NULL, NULL) == PDEC_OK);
    CHECK(pdec_check_lengths(&x, 1, ev_neg, pl_ok, NULL, NULL) == PDEC_ERR_BAD_LENGTHS);
    CHECK(pdec_check_lengths(&x, 1, ev_big, pl_ok, NULL, NULL) == PDEC_ERR_BAD_LENGTHS);
    CHECK(pdec_check_lengths(&x, 1, ev_ok, pl_big, NULL, NULL) == PDEC_ERR_BAD_LENGTHS);
    CHECK(pdec_check_lengths(&x, 1, ev_ok, pl_neg, NULL, NULL) == PDEC_ERR_BAD_LENGTHS);
    CHECK(pdec_check_lengths(&x, 1, NULL, pl_ok, NULL, NULL) == PDEC_ERR_INVALID_ARG);
    CHECK(pdec_check_lengths(&x, 1, ev_ok, NULL, NULL, NULL) == PDEC_ERR_INVALID_ARG);
    const int32_t cp_ok[3] = {0, 100, 150}, ce_ok[3] = {0, 2, 4};
    const int32_t cp_down[3] = {0, 100, 90}, cp_sum[3] = {0, 100, 149}, ce_many[3] = {0, 4, 4}, ce_end[3] = {0, 2, 3};
    CHECK(pdec_check_lengths(&x, 2, ev_ok, NULL, cp_ok, ce_ok) == PDEC_OK);
    CHECK(pdec_check_lengths(&x, 2, ev_ok, NULL, cp_down, ce_ok) == PDEC_ERR_BAD_LENGTHS);
    CHECK(pdec_check_lengths(&x, 2, ev_ok, NULL, cp_sum, ce_ok) == PDEC_ERR_BAD_LENGTHS);
    CHECK(pdec_check_lengths(&x, 2, ev_ok, NULL, cp_ok, ce_many) == PDEC_ERR_BAD_LENGTHS);
    CHECK(pdec_check_lengths(&x, 2, ev_ok, NULL, cp_ok, ce_end) == PDEC_ERR_BAD_LENGTHS);
    CHECK(pdec_check_lengths(&x, 2, ev_ok, NULL, NULL, ce_ok) == PDEC_ERR_INVALID_ARG);
    CHECK(pdec_check_lengths(NULL, 1, ev_ok, pl_ok, NULL, NULL) != PDEC_OK);
    return 0;
}

static int refusals(void)
{
    pdec_dims x = dims(32, 28, 4, 128, 129, 32768, PDEC_DTYPE_BF16);
    const size_t ws = pdec_workspace_size(&x, 1);
    CHECK(ws > 0);
    /* null and misaligned pointers, a short workspace */
    CHECK(pdec_attn_step(&x, NULL, FAKE(1), FAKE(2), FAKE(3), FAKE(4), FAKE(5), FAKE(6), FAKE(7), NULL, FAKE(8), ws,
                         NULL) == PDEC_ERR_INVALID_ARG);
    CHECK(pdec_attn_step(&x, (char*)FAKE(9) + 2, FAKE(1), FAKE(2), FAKE(3), FAKE(4), FAKE(5), FAKE(6), FAKE(7), NULL,
                         FAKE(8), ws, NULL) == PDEC_ERR_INVALID_ARG);
    CHECK(pdec_attn_step(&x, FAKE(9), FAKE(1), FAKE(2), FAKE(3), FAKE(4), FAKE(5), FAKE(6), FAKE(7), NULL, FAKE(8),
                         ws - 1, NULL) == PDEC_ERR_WORKSPACE);
    CHECK(pdec_attn_step_ragged(&x, 2, FAKE(9), FAKE(1), FAKE(2), NULL, FAKE(3), FAKE(4), FAKE(5), FAKE(6), FAKE(7),
                                NULL, FAKE(8), ws, NULL) == PDEC_ERR_INVALID_ARG);
    CHECK(pdec_attn_step_noalloc(&x, NULL, FAKE(1), FAKE(2), FAKE(3), FAKE(4), FAKE(5), FAKE(6), FAKE(7), NULL,
                                 NULL) == PDEC_ERR_INVALID_ARG);
    CHECK(pdec_kv_append(&x, NULL, FAKE(1), FAKE(2), FAKE(3), FAKE(4), NULL, NULL) == PDEC_ERR_INVALID_ARG);
    /* fused append: counts in and out in one array, a missing new row, half a batch table */
    CHECK(pdec_decode_step(&x, 1, FAKE(1), FAKE(2), FAKE(3), FAKE(4), NULL, NULL, FAKE(5), FAKE(6), FAKE(7), FAKE(8),
                           FAKE(9), FAKE(9), NULL, FAKE(10), NULL, FAKE(11), ws, NULL) == PDEC_ERR_INVALID_ARG);
    CHECK(pdec_decode_step(&x, 1, FAKE(1), FAKE(2), FAKE(3), FAKE(4), NULL, NULL, NULL, FAKE(6), FAKE(7), FAKE(8),
                           FAKE(9), FAKE(12), NULL, FAKE(10), NULL, FAKE(11), ws, NULL) == PDEC_ERR_INVALID_ARG);
    CHECK(pdec_decode_step(&x, 2, FAKE(1), FAKE(2), FAKE(3), NULL, FAKE(13), NULL, FAKE(5), FAKE(6), FAKE(7), FAKE(8),
                           FAKE(9), FAKE(12), NULL, FAKE(10), NULL, FAKE(11), ws, NULL) == PDEC_ERR_INVALID_ARG);
    CHECK(pdec_rope_kv_append(&x, 1, FAKE(1), NULL, FAKE(2), FAKE(3), FAKE(4), FAKE(5), NULL, NULL, FAKE(6), 10000.f,
                              NULL) == PDEC_ERR_INVALID_ARG);
    CHECK(pdec_read_probe(NULL, FAKE(1), 64, 4, 576, 0, FAKE(2), NULL) == PDEC_ERR_INVALID_ARG);
    CHECK(pdec_read_probe(FAKE(1), FAKE(2), 64, 4, 100, 1, FAKE(3), NULL) == PDEC_ERR_INVALID_ARG);
    /* path and timer settings */
    for (int p = 0; p <= 3; ++p) CHECK(pdec_set_path(p) >= 0);
    CHECK(pdec_set_path(4) == PDEC_ERR_INVALID_ARG);
    CHECK(pdec_set_path(-1) == PDEC_ERR_INVALID_ARG);
    CHECK(pdec_set_path(0) >= 0);
    CHECK(pdec_set_split_timer(NULL, NULL, 0) == PDEC_OK);
    CHECK(pdec_set_split_timer(NULL, NULL, -1) != PDEC_OK);
    /* the other kernels' sizing and refusals */
    pdec_ground_dims gd = {8, 1000, 16, 128, PDEC_DTYPE_BF16};
    CHECK(pdec_grounding_workspace_size(&gd) > 0);
    gd.dim = 100;
    CHECK(pdec_grounding_workspace_size(&gd) == 0);
    pdec_aggr_dims ad;
    memset(&ad, 0, sizeof(ad));
    ad.num_events = 8; ad.num_tokens = 1000; ad.num_segments = 16; ad.hidden = 3584;
    ad.mode = PDEC_AGGR_UNIFORM; ad.dtype = PDEC_DTYPE_BF16;
    CHECK(pdec_aggregation_workspace_size(&ad) > 0);
    ad.hidden = 3585;
    CHECK(pdec_aggregation_workspace_size(&ad) == 0);
    pdec_dims bx = dims(4, 8, 2, 128, 48, 1024, PDEC_DTYPE_BF16);
    bx.queries_per_stream = 48;
    CHECK(pdec_backward_workspace_size(&bx) > 0);
    bx.head_dim = 96;
    CHECK(pdec_backward_workspace_size(&bx) == 0);
    /* every status has a text */
    for (int c = -8; c <= 1; ++c) CHECK(pdec_strerror(c) != NULL && pdec_strerror(c)[0] != '\0');
    return 0;
}

int main(void)
{
    if (planner_sweep() || lengths() || refusals()) return 1;
    printf("host sanitizer driver: ok\n");
    return 0;
}
