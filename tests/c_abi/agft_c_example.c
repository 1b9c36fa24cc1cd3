/*
 * agft_c_example.c -- a plain C caller of the tuner ABI (include/agft.h).
 *
 * It owns every device buffer, creates one handle on the null stream, runs T
 * decisions for B instances with contexts from a fixed linear congruential
 * generator and a reward that depends on the chosen arm, flushes, and writes
 * everything it saw to a binary file:
 *   int32 header {B, K, d, T}, then per step t: float ctx[B][d],
 *   int32 action[B], float reward[B].
 * A GPU test replays that record through the Python binding and the oracle.
 *
 * usage: agft_c_example B K d T out.bin
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "agft.h"

#define CHECK_HIP(x) do { hipError_t e_ = (x); if (e_ != hipSuccess) { \
    fprintf(stderr, "HIP error %d at line %d\n", (int)e_, __LINE__); return 2; } } while (0)
#define CHECK_AGFT(x) do { int c_ = (x); if (c_ != AGFT_OK) { \
    fprintf(stderr, "agft error %s at line %d\n", agft_strerror(c_), __LINE__); return 3; } } while (0)

static unsigned long long lcg_state = 2508174417ULL;

/* uniform in [-1, 1) from a 64-bit linear congruential generator */
static float lcg_uniform(void)
{
    lcg_state = lcg_state * 6364136223846793005ULL + 1442695040888963407ULL;
    return (float)((lcg_state >> 40) & 0xFFFFFF) / 8388608.0f - 1.0f;
}

int main(int argc, char **argv)
{
    if (argc != 6) {
        fprintf(stderr, "usage: %s B K d T out.bin\n", argv[0]);
        return 1;
    }
    const int B = atoi(argv[1]), K = atoi(argv[2]), d = atoi(argv[3]), T = atoi(argv[4]);
    FILE *out = fopen(argv[5], "wb");
    if (out == NULL || B < 1 || K < 1 || T < 1) return 1;

    agft_config cfg;
    memset(&cfg, 0, sizeof(cfg));
    cfg.B = B;
    cfg.K = K;
    cfg.d = d;
    cfg.lambda = 1.0f;
    cfg.alpha0 = 0.5f;
    cfg.alpha_sched = 0;
    cfg.prune_rule = 1;
    cfg.prune_period = 10;
    cfg.prune_sticky = 1;
    const size_t nbytes = agft_state_bytes(&cfg);
    if (nbytes == 0) {
        fprintf(stderr, "invalid configuration\n");
        return 1;
    }
    if (agft_abi_version() != AGFT_ABI_VERSION) {
        fprintf(stderr, "library ABI %d, header %d\n", agft_abi_version(), AGFT_ABI_VERSION);
        return 1;
    }

    void *d_state = NULL;
    float *d_ctx = NULL, *d_reward = NULL;
    int32_t *d_action = NULL;
    CHECK_HIP(hipMalloc(&d_state, nbytes));
    CHECK_HIP(hipMalloc((void **)&d_ctx, sizeof(float) * B * d));
    CHECK_HIP(hipMalloc((void **)&d_reward, sizeof(float) * B));
    CHECK_HIP(hipMalloc((void **)&d_action, sizeof(int32_t) * B));

    agft_handle *h = NULL;
    CHECK_AGFT(agft_create(&cfg, d_state, nbytes, NULL, &h));

    float *ctx = (float *)malloc(sizeof(float) * B * d);
    float *reward = (float *)malloc(sizeof(float) * B);
    int32_t *action = (int32_t *)malloc(sizeof(int32_t) * B);
    const int32_t header[4] = {B, K, d, T};
    fwrite(header, sizeof(int32_t), 4, out);

    for (int t = 0; t < T; ++t) {
        for (int i = 0; i < B; ++i) {
            ctx[i * d] = 1.0f;
            for (int q = 1; q < d; ++q) ctx[i * d + q] = lcg_uniform();
        }
        CHECK_HIP(hipMemcpy(d_ctx, ctx, sizeof(float) * B * d, hipMemcpyHostToDevice));
        /* the reward of the previous decision is already in d_reward (t > 0) */
        CHECK_AGFT(agft_step(h, d_ctx, t > 0 ? d_reward : NULL, d_action, NULL));
        CHECK_HIP(hipMemcpy(action, d_action, sizeof(int32_t) * B, hipMemcpyDeviceToHost));
        for (int i = 0; i < B; ++i) {
            /* best arm near 0.3 K, plus a context term and noise */
            const float a = (float)action[i] / (float)(K > 1 ? K - 1 : 1);
            reward[i] = -1.0f - 2.0f * (a - 0.3f) * (a - 0.3f) + 0.2f * ctx[i * d + 1]
                        + 0.05f * lcg_uniform();
        }
        CHECK_HIP(hipMemcpy(d_reward, reward, sizeof(float) * B, hipMemcpyHostToDevice));
        fwrite(ctx, sizeof(float), (size_t)B * d, out);
        fwrite(action, sizeof(int32_t), (size_t)B, out);
        fwrite(reward, sizeof(float), (size_t)B, out);
    }
    CHECK_AGFT(agft_step(h, NULL, d_reward, NULL, NULL));   /* flush the last reward */
    CHECK_HIP(hipDeviceSynchronize());

    agft_state_view v;
    CHECK_AGFT(agft_get_state(h, &v));
    printf("steps %lld pending %d instances %d arms %d\n", (long long)v.t, v.pending, v.B, v.K);
    CHECK_AGFT(agft_destroy(h));
    fclose(out);
    free(ctx);
    free(reward);
    free(action);
    hipFree(d_state);
    hipFree(d_ctx);
    hipFree(d_reward);
    hipFree(d_action);
    return 0;
}
