/*
 * Calls the host-side entry points of libagft that enqueue nothing
 * (sizes, launch shapes, argument checks, status strings) over valid,
 * extreme and invalid configurations, so that a host build with the
 * address and undefined-behaviour sanitizers can check the validation and
 * layout arithmetic.  Needs no GPU.  Test infrastructure only.
 */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "agft.h"
#include "agft_sim.h"

static agft_config base(int B, int K, int d)
{
    agft_config c;
    memset(&c, 0, sizeof(c));
    c.B = B;
    c.K = K;
    c.d = d;
    c.lambda = 1.0f;
    c.alpha0 = 0.5f;
    c.prune_rule = 1;
    c.prune_period = 50;
    c.prune_sticky = 1;
    return c;
}

int main(void)
{
    int fails = 0;
    const int dims[] = {8, 16, 32, 12};
    const int arms[] = {1, 2, 27, 63, 64, 65, 128, 129, 1023, 1024, 1025};
    const int batches[] = {1, 3, 4096, 65536, 1 << 20};
    for (unsigned a = 0; a < sizeof(dims) / sizeof(dims[0]); ++a)
        for (unsigned b = 0; b < sizeof(arms) / sizeof(arms[0]); ++b)
            for (unsigned c = 0; c < sizeof(batches) / sizeof(batches[0]); ++c)
                for (int variant = 0; variant < 6; ++variant) {
                    agft_config cfg = base(batches[c], arms[b], dims[a]);
                    if (variant == 1) {
                        cfg.prune_rule = 15;
                        cfg.ext_rounds = 60; cfg.ext_min_n = 3; cfg.ext_thr = -1.2f;
                        cfg.hist_after = 30; cfg.hist_min_n = 6; cfg.hist_kappa = 1.0f;
                        cfg.hist_min_arms = 3; cfg.cascade_k = arms[b] / 3;
                    }
                    if (variant == 2) {
                        cfg.exploit = 1; cfg.ph_delta = 0.05f; cfg.ph_lambda = 5.0f;
                        cfg.ph_window = 100; cfg.ph_min_rounds = 100;
                    }
                    if (variant == 3) {
                        cfg.refine = 1; cfg.refine_period = 50; cfg.refine_stride = 10;
                        cfg.refine_half = 10; cfg.refine_mature = 100; cfg.refine_min_n = 4;
                    }
                    if (variant == 4) cfg.prune_sticky = 0;
                    if (variant == 5) { cfg.prune_sticky = 0; cfg.prune_rule = 3; cfg.ext_min_n = 1; }
                    const size_t n = agft_state_bytes(&cfg);
                    agft_launch_shape shape;
                    const int rc = agft_launch_shape_for(&cfg, &shape);
                    const int valid = dims[a] != 12 && arms[b] <= 1024 && variant != 5;
                    if ((n != 0) != valid || (rc == AGFT_OK) != valid) {
                        printf("unexpected: d=%d K=%d B=%d variant %d: bytes %zu, shape %d\n", dims[a], arms[b],
                               batches[c], variant, n, rc);
                        ++fails;
                    }
                    agft_handle *h = (agft_handle *)0x1;
                    if (agft_create(&cfg, NULL, n, NULL, &h) != AGFT_E_INVAL || h != NULL) ++fails;
                    /* a misaligned buffer: refused, unless the configuration already was */
                    const int unsupported = arms[b] <= 1024 && (dims[a] == 12 || variant == 5);
                    const int want = unsupported ? AGFT_E_UNSUPPORTED : AGFT_E_INVAL;
                    if (agft_create(&cfg, (void *)0x1001, n, NULL, &h) != want) {
                        printf("create: d=%d K=%d variant %d\n", dims[a], arms[b], variant);
                        ++fails;
                    }
                }
    agft_config bad = base(4, 16, 8);
    bad.lambda = 0.0f;
    if (agft_state_bytes(&bad) != 0 || agft_state_bytes(NULL) != 0) ++fails;
    if (agft_launch_shape_for(&bad, NULL) != AGFT_E_INVAL) ++fails;
    if (agft_step(NULL, NULL, NULL, NULL, NULL) != AGFT_E_INVAL) ++fails;
    if (agft_export(NULL, NULL, NULL) != AGFT_E_INVAL || agft_set_stream(NULL, NULL) != AGFT_E_INVAL) ++fails;
    agft_state_view view;
    if (agft_get_state(NULL, &view) != AGFT_E_INVAL || agft_destroy(NULL) != AGFT_OK) ++fails;
    for (int code = -6; code <= 1; ++code)
        if (agft_strerror(code) == NULL || strlen(agft_strerror(code)) == 0) ++fails;
    if (agft_abi_version() != AGFT_ABI_VERSION) ++fails;
    agft_env_config env;
    memset(&env, 0, sizeof(env));
    env.B = 8; env.K = 16; env.d = 8; env.T = 10;
    if (agft_env_state_bytes(&env) != 0) ++fails;   /* zero floors and deviations: invalid */
    if (agft_env_state_bytes(NULL) != 0) ++fails;
    if (agft_sim_step(NULL, &env, NULL, 0, NULL, NULL, NULL, NULL, NULL, NULL) != AGFT_E_INVAL) ++fails;
    printf("abi driver: %d failures\n", fails);
    return fails != 0;
}
