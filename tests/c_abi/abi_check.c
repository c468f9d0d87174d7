/*
 * A plain-C consumer of librevisit, built with gcc as C11 against
 * include/revisit.h (the header must be valid C, the library callable without
 * C++ or Python).
 *
 *   abi_check        host only: status strings, and the host-side argument
 *                    validation of every entry point. Each call below fails
 *                    validation, so it returns before any device call.
 *   abi_check --gpu  also runs, on hipMalloc'd device buffers, the identity
 *                    case of both correspondence calls (Sec. 4.3): with
 *                    the target pose and intrinsics repeated as the source, every
 *                    token maps onto itself, so every code is the token's own
 *                    index. For reproject_correspondence this needs a
 *                    constant positive depth, which also passes Eq. visibility.
 *
 * Exit status 0 when every check passes; otherwise the first failing check
 * is printed and the status is 1.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "revisit.h"

static int failures = 0;

#define CHECK(cond, ...)                                  \
    do {                                                  \
        if (!(cond)) {                                    \
            fprintf(stderr, "FAILED %s:%d: ", __FILE__, __LINE__); \
            fprintf(stderr, __VA_ARGS__);                 \
            fprintf(stderr, "\n");                        \
            failures++;                                   \
        }                                                 \
    } while (0)

/* a non-NULL address that validation rejects before it could be used */
#define FAKE ((void*)0x1000)

static void host_checks(void) {
    CHECK(strcmp(rc_status_string(REVISIT_OK), "ok") == 0, "status string of REVISIT_OK");
    CHECK(strlen(rc_status_string(REVISIT_ERR_NULL)) > 0, "status string of REVISIT_ERR_NULL");

    int st = retrieve_chunks(NULL, 10, FAKE, FAKE, 1, 1.0f, 0.5f, 0.1f, 0.5f, 3, 1, 4, FAKE, NULL, FAKE, 0, NULL,
                             NULL, 0, NULL);
    CHECK(st == REVISIT_ERR_NULL, "retrieve_chunks with a NULL bank: %d", st);
    CHECK(strlen(rc_last_error()) > 0, "rc_last_error after a failure");

    /* workspace sizes: 2 queries x 64 segments of 16384 entries x k = 4 x 12 bytes */
    size_t bytes = 1;
    st = rc_retrieve_workspace_size(1 << 20, 2, 4, &bytes);
    CHECK(st == REVISIT_OK && bytes == (size_t)2 * 64 * 4 * 12, "retrieval workspace of a 2^20 bank: %d, %zu", st,
          bytes);
    st = rc_retrieve_workspace_size(8192, 2, 4, &bytes);
    CHECK(st == REVISIT_OK && bytes == 0, "retrieval workspace of an 8192-entry bank: %d, %zu", st, bytes);
    st = retrieve_chunks(FAKE, 1 << 20, FAKE, FAKE, 2, 1.0f, 0.5f, 0.1f, 0.5f, 3, 1, 4, FAKE, NULL, FAKE, 0, NULL,
                         NULL, 0, NULL);
    CHECK(st == REVISIT_ERR_SHAPE, "retrieve_chunks over a 2^20 bank without a workspace: %d", st);
    /* 37 query tiles x 12 heads = 444 items, 4 parts of 128 x 128 + 2 x 128 floats */
    st = rc_attention_workspace_size(REVISIT_BF16, 4680, 37440, 12, 128, 4, &bytes);
    CHECK(st == REVISIT_OK && bytes == (size_t)444 * 4 * 16640 * 4, "attention workspace in 4 parts: %d, %zu", st,
          bytes);
    st = rc_attention_workspace_size(REVISIT_BF16, 4680, 37440, 12, 128, 1, &bytes);
    CHECK(st == REVISIT_OK && bytes == 0, "attention workspace in 1 part: %d, %zu", st, bytes);
    st = rc_attention_workspace_size(REVISIT_F32, 4680, 37440, 12, 128, 4, &bytes);
    CHECK(st == REVISIT_OK && bytes == 0, "fp32 attention workspace: %d, %zu", st, bytes);
    st = rc_attention_workspace_size(REVISIT_BF16, 4680, 37440, 12, 128, 65, &bytes);
    CHECK(st == REVISIT_ERR_PARAM, "attention workspace with 65 key parts: %d", st);
    st = biased_chunk_attention(FAKE, FAKE, FAKE, FAKE, NULL, REVISIT_BF16, 4680, 37440, 12, 128, 30, 52, FAKE, FAKE,
                                FAKE, 12, 0.088f, 1.0f, 2.0f, 4, FAKE, 4096, NULL);
    CHECK(st == REVISIT_ERR_SHAPE, "biased_chunk_attention with a 4 KiB workspace for 4 key parts: %d", st);
    /* 64 parts of 444 items need 1.9 GB of partial results, more than the no-allocation scratch */
    st = biased_chunk_attention_noalloc(FAKE, FAKE, FAKE, FAKE, NULL, REVISIT_BF16, 4680, 37440, 12, 128, 30, 52, FAKE,
                                        FAKE, FAKE, 12, 0.088f, 1.0f, 2.0f, 64, NULL);
    CHECK(st == REVISIT_ERR_SHAPE, "biased_chunk_attention_noalloc with 64 key parts: %d", st);

    st = reproject_correspondence(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, NULL, 0, 1, 3, 6, 30, 52, 2, -1.0f, FAKE, FAKE,
                                  NULL);
    CHECK(st == REVISIT_ERR_PARAM, "reproject_correspondence with eps < 0: %d", st);

    st = reproject_rotation(NULL, FAKE, FAKE, FAKE, NULL, 0, 1, 3, 6, 30, 52, 2, FAKE, FAKE, NULL);
    CHECK(st == REVISIT_ERR_NULL, "reproject_rotation with a NULL target pose: %d", st);
    st = reproject_rotation(FAKE, FAKE, FAKE, FAKE, NULL, 0, 1, 3, 65, 30, 52, 2, FAKE, FAKE, NULL);
    CHECK(st == REVISIT_ERR_SHAPE, "reproject_rotation with 65 sources: %d", st);

    st = biased_chunk_attention(FAKE, FAKE, FAKE, FAKE, NULL, REVISIT_BF16, 4680, 28080, 12, 128, 30, 52, FAKE, FAKE,
                                FAKE, 6, 0.088f, 1.0f, 0.0f, 0, NULL, 0, NULL);
    CHECK(st == REVISIT_ERR_PARAM, "biased_chunk_attention with sigma = 0: %d", st);

    st = pack_retrieved_kv(FAKE, FAKE, NULL, 200, FAKE, 4, 3, NULL, FAKE, 4680, 37440, 30, REVISIT_BF16, 3, 30, 52, 12,
                           128, 22, 10000.0f, NULL);
    CHECK(st == REVISIT_ERR_NULL, "pack_retrieved_kv with a NULL cache: %d", st);

    st = pool_token_depth(NULL, 2, 30, 52, 2, FAKE, NULL);
    CHECK(st == REVISIT_ERR_NULL, "pool_token_depth with a NULL depth map: %d", st);

    rc_stream* s = NULL;
    st = rc_stream_create(NULL, &s);
    CHECK(st == REVISIT_ERR_NULL && s == NULL, "rc_stream_create without a configuration: %d", st);
}

/* one problem: Tq = 1 target frame, S = 2 sources, an h x w grid at p = 2 */
enum { H_TOK = 9, W_TOK = 13, P = 2, S_SRC = 2 };

static int gpu_checks(void) {
    const int n = H_TOK * W_TOK, hd = H_TOK * P, wd = W_TOK * P;
    float pose[16] = {0.8f, -0.6f, 0.0f, 1.5f, 0.6f, 0.8f, 0.0f, -2.0f, 0.0f, 0.0f, 1.0f, 0.25f, 0, 0, 0, 1};
    float K[4] = {20.0f, 20.0f, 13.0f, 9.0f};
    float h_c2w[16 * (1 + S_SRC)], h_K[4 * (1 + S_SRC)];
    for (int f = 0; f < 1 + S_SRC; ++f) {
        memcpy(h_c2w + 16 * f, pose, sizeof pose);
        memcpy(h_K + 4 * f, K, sizeof K);
    }
    float* h_depth = (float*)malloc(sizeof(float) * (1 + S_SRC) * hd * wd);
    for (int i = 0; i < (1 + S_SRC) * hd * wd; ++i) h_depth[i] = 4.0f;

    float *d_c2w = NULL, *d_K = NULL, *d_depth = NULL, *d_uv = NULL;
    int32_t* d_idx = NULL;
    if (hipMalloc((void**)&d_c2w, sizeof h_c2w) != hipSuccess || hipMalloc((void**)&d_K, sizeof h_K) != hipSuccess ||
        hipMalloc((void**)&d_depth, sizeof(float) * (1 + S_SRC) * hd * wd) != hipSuccess ||
        hipMalloc((void**)&d_uv, sizeof(float) * 2 * S_SRC * n) != hipSuccess ||
        hipMalloc((void**)&d_idx, sizeof(int32_t) * S_SRC * n) != hipSuccess) {
        fprintf(stderr, "hipMalloc failed\n");
        return 1;
    }
    hipMemcpy(d_c2w, h_c2w, sizeof h_c2w, hipMemcpyHostToDevice);
    hipMemcpy(d_K, h_K, sizeof h_K, hipMemcpyHostToDevice);
    hipMemcpy(d_depth, h_depth, sizeof(float) * (1 + S_SRC) * hd * wd, hipMemcpyHostToDevice);

    int32_t* h_idx = (int32_t*)malloc(sizeof(int32_t) * S_SRC * n);
    for (int call = 0; call < 2; ++call) {
        hipMemset(d_idx, 0xff, sizeof(int32_t) * S_SRC * n);
        int st;
        if (call == 0) {
            fprintf(stderr, "abi_check: reproject_correspondence identity %dx%d p=%d\n", H_TOK, W_TOK, P);
            st = reproject_correspondence(d_depth, d_c2w, d_K, d_depth + hd * wd, d_c2w + 16, d_K + 4, NULL, 0, 1, 1,
                                          S_SRC, H_TOK, W_TOK, P, 0.05f, d_uv, d_idx, NULL);
        } else {
            fprintf(stderr, "abi_check: reproject_rotation identity %dx%d p=%d\n", H_TOK, W_TOK, P);
            st = reproject_rotation(d_c2w, d_K, d_c2w + 16, d_K + 4, NULL, 0, 1, 1, S_SRC, H_TOK, W_TOK, P, d_uv,
                                    d_idx, NULL);
        }
        CHECK(st == REVISIT_OK, "call %d returned %d (%s)", call, st, rc_last_error());
        CHECK(hipDeviceSynchronize() == hipSuccess, "synchronise after call %d", call);
        hipMemcpy(h_idx, d_idx, sizeof(int32_t) * S_SRC * n, hipMemcpyDeviceToHost);
        int bad = 0;
        for (int s = 0; s < S_SRC; ++s)
            for (int t = 0; t < n; ++t) bad += h_idx[s * n + t] != t;
        CHECK(bad == 0, "call %d: %d tokens not mapped onto themselves", call, bad);
    }
    free(h_idx);
    free(h_depth);
    hipFree(d_c2w);
    hipFree(d_K);
    hipFree(d_depth);
    hipFree(d_uv);
    hipFree(d_idx);
    return 0;
}

int main(int argc, char** argv) {
    host_checks();
    if (argc > 1 && strcmp(argv[1], "--gpu") == 0) {
        if (gpu_checks() != 0) return 1;
    }
    if (failures) return 1;
    printf("abi_check: ok\n");
    return 0;
}
