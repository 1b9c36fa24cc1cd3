/*
 * Drives the fp64 oracle (oracle/agft_oracle.c, compiled into this program)
 * through every option it has, so that a build with the address and
 * undefined-behaviour sanitizers can check its memory accesses and
 * arithmetic: confidence-bound pruning (sticky and re-evaluated), the
 * paper's rules 2-8, the exploitation switch, the refinement, non-finite
 * contexts and rewards, the accessors, flush and destroy.  Test
 * infrastructure only.  Exits 0 when every run completed.
 */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

#include "../../oracle/agft_oracle.c"

static unsigned long long rng_state = 0x2508174425081744ull;

static double uniform(void)
{
    rng_state = rng_state * 6364136223846793005ull + 1442695040888963407ull;
    return (double)(rng_state >> 11) / 9007199254740992.0;
}

static int run(int B, int K, int d, int prune, int period, int sched, int sticky, int rules, int exploit,
               int refine, int T, int bad_inputs)
{
    void *h = ora_create(B, K, d, 1.0, 0.6, sched, prune | rules, period);
    if (!h) return 1;
    ora_set_sticky(h, sticky);
    if (rules) ora_set_heuristics(h, 40, 2, -1.1, 10, 3, 0.8, 3, K / 3);
    if (exploit) ora_set_exploit(h, 1, 0.05, 2.0, 15, 20);
    if (refine) ora_set_refine(h, 1, 7, 4, 3, 30, 2);
    double *x = malloc(sizeof(double) * B * d), *r = malloc(sizeof(double) * B);
    double *ucb = malloc(sizeof(double) * B * K), *lcb = malloc(sizeof(double) * B * K);
    double *marg = malloc(sizeof(double) * B * K);
    unsigned char *keep = malloc((size_t)B * K);
    int *action = malloc(sizeof(int) * B);
    double *A = malloc(sizeof(double) * K * d * d), *b = malloc(sizeof(double) * K * d);
    double *Ainv = malloc(sizeof(double) * K * d * d), *theta = malloc(sizeof(double) * K * d);
    double *rsum = malloc(sizeof(double) * K), *stats = malloc(sizeof(double) * 6 * B);
    double *margins = malloc(sizeof(double) * B);
    long *last = malloc(sizeof(long) * B), *mode = malloc(sizeof(long) * B);
    int *win = malloc(sizeof(int) * 3 * B), *nsel = malloc(sizeof(int) * K);
    unsigned char *active = malloc((size_t)K);
    int pending = 0;
    for (int t = 0; t < T; ++t) {
        for (int i = 0; i < B; ++i) {
            x[i * d] = 1.0;
            for (int q = 1; q < d; ++q) x[i * d + q] = 2.0 * uniform() - 1.0;
            r[i] = -2.0 * uniform();
        }
        if (bad_inputs && t % 9 == 4) x[(t % B) * d + 1] = NAN;
        if (bad_inputs && t % 11 == 6) r[(t + 1) % B] = INFINITY;
        ora_decide_ex(h, x, pending ? r : NULL, ucb, lcb, keep, action, marg);
        ora_commit(h, x, action, keep);
        pending = 1;
        ora_get_ph_all(h, stats, margins, last, mode);
        ora_get_window_all(h, win);
    }
    ora_flush(h, r);
    for (int i = 0; i < B; ++i) {
        int bad = 0;
        ora_get(h, i, A, b, Ainv, theta, active, nsel, &bad);
        ora_get_rsum(h, i, rsum);
        double st[6], m;
        long l, mo;
        int lo, hi, stride;
        ora_get_ph(h, i, st, &m, &l, &mo);
        ora_set_ph(h, i, st, m, l, mo);
        ora_get_window(h, i, &lo, &hi, &stride);
        ora_set_window(h, i, lo, hi, stride);
    }
    (void)ora_alpha(h, T);
    (void)ora_t_now(h);
    ora_destroy(h);
    free(x); free(r); free(ucb); free(lcb); free(marg); free(keep); free(action); free(A); free(b);
    free(Ainv); free(theta); free(rsum); free(stats); free(margins); free(last); free(mode); free(win);
    free(nsel); free(active);
    return 0;
}

int main(void)
{
    int fails = 0;
    fails += run(3, 5, 1, 0, 5, 0, 1, 0, 0, 0, 30, 0);
    fails += run(4, 16, 8, 1, 6, 0, 1, 0, 0, 0, 80, 1);
    fails += run(3, 40, 16, 1, 5, 1, 0, 0, 1, 1, 90, 1);      /* non-sticky, switch, refinement */
    fails += run(2, 33, 32, 1, 7, 0, 1, 14, 1, 0, 70, 1);     /* rules 2-8 and the switch */
    fails += run(2, 100, 8, 1, 9, 0, 1, 14, 0, 1, 70, 0);     /* rules with the refinement */
    fails += run(1, 1024, 4, 1, 10, 0, 0, 0, 0, 0, 25, 1);    /* the largest arm count */
    if (ora_create(0, 4, 4, 1.0, 1.0, 0, 0, 5) != NULL) ++fails;   /* rejected configurations */
    if (ora_create(1, 2000, 4, 1.0, 1.0, 0, 0, 5) != NULL) ++fails;
    if (ora_create(1, 4, 4, -1.0, 1.0, 0, 0, 5) != NULL) ++fails;
    printf("oracle driver: %d failures\n", fails);
    return fails != 0;
}
