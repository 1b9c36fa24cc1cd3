/*
 * agft_oracle.c -- CPU fp64 oracle of the AGFT contextual-bandit step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may load, link or
 * call this file; only the tests, the smoke check and the benchmark's
 * CPU-baseline leg do.  It shares no code, header or constant with the GPU
 * path.
 *
 * What it computes (disjoint LinUCB over the frequency arms, Sec. 4.2), for
 * every tuner instance independently, in double precision:
 *
 *   A_k = lambda I + sum over past steps s with a_s = k of x_s x_s^T   (Eq. 3)
 *   b_k =            sum over past steps s with a_s = k of r_s x_s     (Eq. 4)
 *   theta_k = A_k^{-1} b_k                                             (Eq. 5)
 *   UCB_k = theta_k^T x_t + alpha_t sqrt(x_t^T A_k^{-1} x_t)           (Eq. 1)
 *   LCB_k = theta_k^T x_t - alpha_t sqrt(x_t^T A_k^{-1} x_t)
 *   a_t   = lowest index among the active arms with the largest UCB_k  (Eq. 1)
 *
 * Readings where the paper is silent: A_k starts at lambda I and b_k at 0;
 * alpha_t is alpha0 or alpha0 / sqrt(t + 1); ties go to the lowest arm index;
 * a negative rounding of the quadratic form is taken as 0 under the root.
 *
 * Pruning; every rule removes arms for good (as Sec. 4.3 says of its own rules).
 * The rule set is a bit mask:
 *   1  confidence bounds: at a step t > 0 with t % period == 0, an active arm
 *      k stays active iff UCB_k >= max over the active arms j of LCB_j, all
 *      scores taken with that step's x_t and alpha_t, before the argmax;
 *   2  extreme-frequency pruning (Sec. 4.3): while t < ext_rounds, an active
 *      arm with n_k >= ext_min_n rewards and mean reward below ext_thr goes;
 *   4  historical-performance pruning (Sec. 4.3): once t >= hist_after, among
 *      the active arms with n_k >= hist_min_n (at least hist_min_arms of
 *      them) an arm goes when the best of their mean rewards exceeds its own
 *      by more than hist_kappa times the (population) standard deviation of
 *      those means;
 *   8  cascade pruning (Sec. 4.3): when rule 2 or 4 removes an arm below
 *      half of the top clock (index < cascade_k), every lower arm goes too.
 * Rules 2-8 act on the arms active at the start of the step, after the
 * previous decision's reward has been folded in and before scoring; rules 2
 * and 4 are judged together.  If they would leave no arm, the one with the
 * best mean reward (lowest index on ties) stays.
 *
 * Non-sticky reading of rule 1 (ora_set_sticky(h, 0); rule 1 alone, no rule
 * 2-8): at each of its steps rule 1 starts again from the whole action
 * space instead of the arms still active, so the kept set is
 * {k in space : UCB_k >= max over the space of LCB_j}, every arm of the space
 * scored; between its steps that set stands.  An arm removed once can come
 * back at a later rule-1 step.
 *
 * The paper gives the update as Eq. 3-5: A and b are accumulated as written
 * and A_k^{-1} is recomputed by Gauss-Jordan elimination with partial
 * pivoting each time A_k changes; theta_k is then recomputed as A_k^{-1} b_k.
 * There is no rank-1 identity here: that is the GPU path's business.
 *
 * Exploitation (Sec. 4.2, Eq. 2), when enabled: each reward folded in also
 * feeds a two-sided Page-Hinkley test on the instance's reward sequence, in
 * double precision like everything else here.  With r_1..r_n the rewards
 * since the test last (re)started and rbar_s the mean of r_1..r_s:
 *   m+_n = sum_{s<=n} (r_s - rbar_s - delta),  M+_n = min(0, m+_1, ..., m+_n),
 *   m-_n = sum_{s<=n} (rbar_s - r_s - delta),  M-_n = min(0, m-_1, ..., m-_n);
 * an alarm is raised when m+_n - M+_n or m-_n - M-_n exceeds lambda, and the
 * test restarts (n = 0).  The sequence counts as stable once t >= min_rounds
 * and no alarm was raised in the last `window` rounds; from then on the
 * instance exploits for good: a_t = argmax over the active arms of
 * theta_k^T x_t (reported as both UCB and LCB), rule 1 is not applied,
 * updates go on.
 *
 * Mixed-maturity refinement (Sec. 4.4), when enabled: the action space is a
 * set of arms on the K-arm grid (one arm step plays the paper's 15 MHz),
 * lo <= k <= hi with (hi - k) % stride == 0, intersected with the arms no
 * pruning rule has removed.  It starts as the coarse grid lo = 0, hi = K-1,
 * stride = refine_stride.  At a step t > 0 with t % refine_period == 0 that
 * made a decision, after the decision, an anchor is chosen among the arms of
 * the action space that survived this step's pruning: before round
 * refine_mature the one with the best mean reward (the lowest mean EDP)
 * among those with at least refine_min_n rewards (lowest index on ties; no
 * refinement if none qualifies), from then on the arm this step chose (the
 * highest UCB, or theta^T x once exploiting).  The action space becomes the
 * full-resolution window lo = max(0, anchor - refine_half), hi = min(K-1,
 * anchor + refine_half), stride 1, from the next step on.  Every arm keeps
 * its model across refinements; pruned arms stay pruned.
 *
 * Step order: the reward r_{t-1} of the previous decision arrives with the
 * next context, so ora_decide first applies Eq. 3-5 to the arm chosen at
 * t-1 with (x_{t-1}, r_{t-1}), then scores x_t, prunes and picks a_t.
 * ora_commit then records the decision that was taken (the test harness may
 * commit another near-tied arm), and ora_flush applies the last pending
 * update without deciding.
 *
 * Non-finite inputs: a non-finite r_{t-1} skips that update; a non-finite
 * x_t yields action -1 (no decision) and no update next step.  Each such
 * event increments the instance's bad-input counter.
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORA_MAXD 64

/* State of one two-sided Page-Hinkley test (see the header). */
struct ph_test {
    double n;       /* rewards since the last restart */
    double sum;     /* their sum: rbar_n = sum / n */
    double up;      /* m+_n */
    double up_min;  /* M+_n (0 at a restart) */
    double dn;      /* m-_n */
    double dn_min;  /* M-_n */
};

typedef struct {
    int B, K, d, prune, period, sched;
    int sticky;             /* 1: rule 1 removes for good; 0: re-evaluated over the space */
    double lambda, alpha0;
    /* parameters of rules 2-8 */
    int ext_rounds, ext_min_n, hist_after, hist_min_n, hist_min_arms, cascade_k;
    double ext_thr, hist_kappa;
    /* exploitation switch (Page-Hinkley test on the rewards) */
    int exploit, ph_window, ph_min_rounds;
    double ph_delta, ph_lambda;
    struct ph_test *ph;     /* [B]           one test per instance */
    /* mixed-maturity refinement */
    int refine, refine_period, refine_stride, refine_half, refine_mature, refine_min_n;
    int *win;               /* [B][3]        action space lo, hi, stride */
    double *ph_margin;      /* [B]           lambda - larger statistic at the last test */
    long *ph_last;          /* [B]           round of the last alarm (0 at start) */
    long *mode;             /* [B]           -1 exploring, else the round exploitation began */
    double *A;              /* [B][K][d][d]  Eq. 3 */
    double *b;              /* [B][K][d]     Eq. 4 */
    double *Ainv;           /* [B][K][d][d]  inverse of A */
    double *theta;          /* [B][K][d]     Eq. 5 */
    unsigned char *active;  /* [B][K]        arms no pruning rule has removed */
    int *nsel;              /* [B][K]        rewards folded into each arm */
    double *rsum;           /* [B][K]        sum of those rewards */
    double *xprev;          /* [B][d]        context of the last decision */
    int *aprev;             /* [B]           last decision (-1: none) */
    int *bad;               /* [B]           non-finite inputs seen */
    long t;                 /* decisions committed so far */
    int pending;            /* 1 while the last decision awaits its reward */
} ora_t;

/* Inverse of the d x d matrix M by Gauss-Jordan elimination on [M | I]
 * with partial pivoting.  Returns 0, or -1 if M is singular. */
static int gauss_jordan_inverse(int d, const double *M, double *out)
{
    double W[ORA_MAXD][2 * ORA_MAXD];
    for (int r = 0; r < d; ++r)
        for (int c = 0; c < d; ++c) {
            W[r][c] = M[r * d + c];
            W[r][d + c] = (r == c) ? 1.0 : 0.0;
        }
    for (int col = 0; col < d; ++col) {
        int piv = col;
        for (int r = col + 1; r < d; ++r)
            if (fabs(W[r][col]) > fabs(W[piv][col])) piv = r;
        if (W[piv][col] == 0.0) return -1;
        if (piv != col)
            for (int c = 0; c < 2 * d; ++c) {
                double tmp = W[col][c]; W[col][c] = W[piv][c]; W[piv][c] = tmp;
            }
        double p = W[col][col];
        for (int c = 0; c < 2 * d; ++c) W[col][c] /= p;
        for (int r = 0; r < d; ++r) {
            if (r == col) continue;
            double f = W[r][col];
            if (f == 0.0) continue;
            for (int c = 0; c < 2 * d; ++c) W[r][c] -= f * W[col][c];
        }
    }
    for (int r = 0; r < d; ++r)
        for (int c = 0; c < d; ++c) out[r * d + c] = W[r][d + c];
    return 0;
}

void ora_decide_ex(void *h, const double *x, const double *r, double *ucb, double *lcb,
                   unsigned char *keep, int *action, double *margins);
void ora_get_rsum(const void *h, int i, double *rsum);
void ora_set_exploit(void *h, int on, double delta, double lambda, int window, int min_rounds);
void ora_get_ph(const void *h, int i, double *stats, double *margin, long *last, long *mode);
void ora_set_ph(void *h, int i, const double *stats, double margin, long last, long mode);
void ora_set_refine(void *h, int on, int period, int stride, int half, int mature, int min_n);
void ora_get_window(const void *h, int i, int *lo, int *hi, int *stride);
void ora_set_window(void *h, int i, int lo, int hi, int stride);
void ora_get_ph_all(const void *h, double *stats, double *margin, long *last, long *mode);
void ora_get_window_all(const void *h, int *win);

static int all_finite(const double *v, int n)
{
    for (int i = 0; i < n; ++i)
        if (!isfinite(v[i])) return 0;
    return 1;
}

void *ora_create(int B, int K, int d, double lambda, double alpha0, int sched,
                 int prune, int period)
{
    if (B < 1 || K < 1 || K > 1024 || d < 1 || d > ORA_MAXD || !(lambda > 0.0) || period < 1)
        return NULL;
    ora_t *o = (ora_t *)calloc(1, sizeof(ora_t));
    if (!o) return NULL;
    o->B = B; o->K = K; o->d = d; o->lambda = lambda; o->alpha0 = alpha0;
    o->sched = sched; o->prune = prune; o->period = period; o->sticky = 1;
    size_t nk = (size_t)B * K;
    o->A = (double *)calloc(nk * d * d, sizeof(double));
    o->b = (double *)calloc(nk * d, sizeof(double));
    o->Ainv = (double *)calloc(nk * d * d, sizeof(double));
    o->theta = (double *)calloc(nk * d, sizeof(double));
    o->active = (unsigned char *)malloc(nk);
    o->nsel = (int *)calloc(nk, sizeof(int));
    o->rsum = (double *)calloc(nk, sizeof(double));
    o->xprev = (double *)calloc((size_t)B * d, sizeof(double));
    o->aprev = (int *)malloc((size_t)B * sizeof(int));
    o->bad = (int *)calloc((size_t)B, sizeof(int));
    o->ph = (struct ph_test *)calloc((size_t)B, sizeof(struct ph_test));
    o->ph_margin = (double *)malloc((size_t)B * sizeof(double));
    o->ph_last = (long *)calloc((size_t)B, sizeof(long));
    o->mode = (long *)malloc((size_t)B * sizeof(long));
    o->win = (int *)malloc((size_t)B * 3 * sizeof(int));
    if (!o->win || !o->A || !o->b || !o->Ainv || !o->theta || !o->active || !o->nsel || !o->rsum ||
        !o->xprev || !o->aprev || !o->bad || !o->ph || !o->ph_margin || !o->ph_last || !o->mode) {
        free(o->A); free(o->b); free(o->Ainv); free(o->theta); free(o->active);
        free(o->nsel); free(o->rsum); free(o->xprev); free(o->aprev); free(o->bad);
        free(o->ph); free(o->ph_margin); free(o->ph_last); free(o->mode); free(o->win); free(o);
        return NULL;
    }
    /* A_k(0) = lambda I, b_k(0) = 0, hence A_k^{-1}(0) = I / lambda, theta_k(0) = 0. */
    for (size_t k = 0; k < nk; ++k)
        for (int r = 0; r < d; ++r) {
            o->A[(k * d + r) * d + r] = lambda;
            o->Ainv[(k * d + r) * d + r] = 1.0 / lambda;
        }
    memset(o->active, 1, nk);
    for (int i = 0; i < B; ++i) {
        o->aprev[i] = -1;
        o->mode[i] = -1;
        o->ph_margin[i] = INFINITY;
        o->win[3 * i] = 0;
        o->win[3 * i + 1] = K - 1;
        o->win[3 * i + 2] = 1;
    }
    return o;
}

void ora_destroy(void *h)
{
    ora_t *o = (ora_t *)h;
    if (!o) return;
    free(o->A); free(o->b); free(o->Ainv); free(o->theta); free(o->active);
    free(o->nsel); free(o->rsum); free(o->xprev); free(o->aprev); free(o->bad);
    free(o->ph); free(o->ph_margin); free(o->ph_last); free(o->mode); free(o->win); free(o);
}

/* Rule 1 sticky (1, the default) or re-evaluated at each of its steps (0). */
void ora_set_sticky(void *h, int sticky)
{
    ((ora_t *)h)->sticky = sticky ? 1 : 0;
}

/* Refinement: on/off and its parameters (see the header); call before the
 * first decision.  Every instance starts on the coarse grid. */
void ora_set_refine(void *h, int on, int period, int stride, int half, int mature, int min_n)
{
    ora_t *o = (ora_t *)h;
    o->refine = on;
    o->refine_period = period;
    o->refine_stride = stride;
    o->refine_half = half;
    o->refine_mature = mature;
    o->refine_min_n = min_n;
    for (int i = 0; i < o->B; ++i) {
        o->win[3 * i] = 0;
        o->win[3 * i + 1] = o->K - 1;
        o->win[3 * i + 2] = on ? stride : 1;
    }
}

/* Action space of instance i (lo, hi, stride); outputs may be NULL. */
void ora_get_window(const void *h, int i, int *lo, int *hi, int *stride)
{
    const ora_t *o = (const ora_t *)h;
    if (lo) *lo = o->win[3 * i];
    if (hi) *hi = o->win[3 * i + 1];
    if (stride) *stride = o->win[3 * i + 2];
}

/* Overwrite instance i's action space (the parity harness adopts the GPU's
 * where two anchor candidates were within rounding of each other). */
void ora_set_window(void *h, int i, int lo, int hi, int stride)
{
    ora_t *o = (ora_t *)h;
    o->win[3 * i] = lo;
    o->win[3 * i + 1] = hi;
    o->win[3 * i + 2] = stride;
}

/* Arm k is in instance i's action space (before pruning). */
static int in_space(const ora_t *o, int i, int k)
{
    const int lo = o->win[3 * i], hi = o->win[3 * i + 1], st = o->win[3 * i + 2];
    return k >= lo && k <= hi && (hi - k) % st == 0;
}

/* Exploitation switch: on/off and the Page-Hinkley parameters (see the header). */
void ora_set_exploit(void *h, int on, double delta, double lambda, int window, int min_rounds)
{
    ora_t *o = (ora_t *)h;
    o->exploit = on;
    o->ph_delta = delta;
    o->ph_lambda = lambda;
    o->ph_window = window;
    o->ph_min_rounds = min_rounds;
}

/* One reward into instance i's Page-Hinkley test at round t. */
static void page_hinkley(ora_t *o, int i, long t, double r)
{
    struct ph_test *p = o->ph + i;
    p->n += 1.0;
    p->sum += r;
    const double rbar = p->sum / p->n;
    p->up += (r - rbar) - o->ph_delta;
    p->dn += (rbar - r) - o->ph_delta;
    if (p->up < p->up_min) p->up_min = p->up;
    if (p->dn < p->dn_min) p->dn_min = p->dn;
    const double stat = fmax(p->up - p->up_min, p->dn - p->dn_min);
    o->ph_margin[i] = o->ph_lambda - stat;
    if (stat > o->ph_lambda) {
        o->ph_last[i] = t;
        memset(p, 0, sizeof(*p));
    }
}

/* The test state as six numbers: n, rbar_n (0 when n = 0), m+, M+, m-, M-. */
static void ph_export(const struct ph_test *p, double *out)
{
    out[0] = p->n;
    out[1] = p->n > 0.0 ? p->sum / p->n : 0.0;
    out[2] = p->up;
    out[3] = p->up_min;
    out[4] = p->dn;
    out[5] = p->dn_min;
}

/* Page-Hinkley state of instance i: stats[6] (n, mean, m+, min m+, m-, min m-),
 * the last margin, the last alarm round and the mode; outputs may be NULL. */
void ora_get_ph(const void *h, int i, double *stats, double *margin, long *last, long *mode)
{
    const ora_t *o = (const ora_t *)h;
    if (stats) ph_export(o->ph + i, stats);
    if (margin) *margin = o->ph_margin[i];
    if (last) *last = o->ph_last[i];
    if (mode) *mode = o->mode[i];
}

/* Every instance's Page-Hinkley state at once: stats [B][6], margin [B],
 * last alarm round [B], mode [B] (a copy; for the harness's batch checks). */
void ora_get_ph_all(const void *h, double *stats, double *margin, long *last, long *mode)
{
    const ora_t *o = (const ora_t *)h;
    const size_t B = (size_t)o->B;
    for (size_t i = 0; i < B; ++i) ph_export(o->ph + i, stats + 6 * i);
    memcpy(margin, o->ph_margin, sizeof(double) * B);
    memcpy(last, o->ph_last, sizeof(long) * B);
    memcpy(mode, o->mode, sizeof(long) * B);
}

/* Every instance's action space at once: win [B][3] = lo, hi, stride (a copy). */
void ora_get_window_all(const void *h, int *win)
{
    const ora_t *o = (const ora_t *)h;
    memcpy(win, o->win, sizeof(int) * 3 * (size_t)o->B);
}

/* Overwrite instance i's Page-Hinkley state and mode from six numbers in the
 * layout of ora_get_ph (the parity harness adopts the GPU's when an alarm
 * comparison sat within rounding of lambda). */
void ora_set_ph(void *h, int i, const double *stats, double margin, long last, long mode)
{
    ora_t *o = (ora_t *)h;
    struct ph_test *p = o->ph + i;
    p->n = stats[0];
    p->sum = stats[1] * stats[0];
    p->up = stats[2];
    p->up_min = stats[3];
    p->dn = stats[4];
    p->dn_min = stats[5];
    o->ph_margin[i] = margin;
    o->ph_last[i] = last;
    o->mode[i] = mode;
}

/* Parameters of pruning rules 2-8 (see the header). */
void ora_set_heuristics(void *h, int ext_rounds, int ext_min_n, double ext_thr, int hist_after,
                        int hist_min_n, double hist_kappa, int hist_min_arms, int cascade_k)
{
    ora_t *o = (ora_t *)h;
    o->ext_rounds = ext_rounds; o->ext_min_n = ext_min_n; o->ext_thr = ext_thr;
    o->hist_after = hist_after; o->hist_min_n = hist_min_n; o->hist_kappa = hist_kappa;
    o->hist_min_arms = hist_min_arms; o->cascade_k = cascade_k;
}

/* Eq. 3-5 for arm k of instance i with context x and reward r. */
static void update_arm(ora_t *o, int i, int k, const double *x, double r)
{
    const int d = o->d;
    size_t ik = (size_t)i * o->K + k;
    double *A = o->A + ik * d * d, *b = o->b + ik * d;
    double *Ainv = o->Ainv + ik * d * d, *theta = o->theta + ik * d;
    for (int p = 0; p < d; ++p)
        for (int q = 0; q < d; ++q) A[p * d + q] += x[p] * x[q];      /* Eq. 3 */
    for (int p = 0; p < d; ++p) b[p] += r * x[p];                      /* Eq. 4 */
    gauss_jordan_inverse(d, A, Ainv);  /* A is lambda I plus PSD terms: never singular */
    for (int p = 0; p < d; ++p) {                                       /* Eq. 5 */
        double s = 0.0;
        for (int q = 0; q < d; ++q) s += Ainv[p * d + q] * b[q];
        theta[p] = s;
    }
    o->nsel[ik] += 1;
    o->rsum[ik] += r;
}

/* Rules 2-8 for instance i at step t: act1 = arms that stay, from act0.
 * margin[k] = distance of arm k's closest rule-2/4 comparison from its
 * threshold (INFINITY when no such rule applied to it). */
static void heuristic_prune(const ora_t *o, int i, long t, const unsigned char *act0,
                            unsigned char *act1, double *margin)
{
    const int K = o->K;
    const int *n = o->nsel + (size_t)i * K;
    const double *rs = o->rsum + (size_t)i * K;
    unsigned char gone[1024];
    double mean[1024];
    for (int k = 0; k < K; ++k) {
        mean[k] = n[k] > 0 ? rs[k] / n[k] : 0.0;
        gone[k] = 0;
        margin[k] = INFINITY;
    }
    if ((o->prune & 2) && t < o->ext_rounds)
        for (int k = 0; k < K; ++k)
            if (act0[k] && n[k] >= o->ext_min_n) {
                double m = mean[k] - o->ext_thr;
                if (fabs(m) < margin[k]) margin[k] = fabs(m);
                if (m < 0.0) gone[k] = 1;
            }
    if ((o->prune & 4) && t >= o->hist_after) {
        int q = 0;
        double best = -INFINITY, sum = 0.0;
        for (int k = 0; k < K; ++k)
            if (act0[k] && n[k] >= o->hist_min_n) {
                ++q;
                sum += mean[k];
                if (mean[k] > best) best = mean[k];
            }
        if (q >= o->hist_min_arms && q > 0) {
            double mu = sum / q, var = 0.0;
            for (int k = 0; k < K; ++k)
                if (act0[k] && n[k] >= o->hist_min_n) var += (mean[k] - mu) * (mean[k] - mu);
            double sigma = sqrt(var / q);
            for (int k = 0; k < K; ++k)
                if (act0[k] && n[k] >= o->hist_min_n) {
                    double m = o->hist_kappa * sigma - (best - mean[k]);
                    if (fabs(m) < margin[k]) margin[k] = fabs(m);
                    if (m < 0.0) gone[k] = 1;
                }
        }
    }
    if (o->prune & 8) {
        int kstar = -1;
        for (int k = 0; k < K; ++k)
            if (gone[k] && k < o->cascade_k) kstar = k;
        for (int k = 0; k < kstar; ++k) gone[k] = 1;
    }
    int left = 0;
    for (int k = 0; k < K; ++k) {
        act1[k] = act0[k] && !gone[k];
        left += act1[k];
    }
    if (left == 0) {
        int keep = -1;
        for (int k = 0; k < K; ++k)
            if (act0[k] && (keep < 0 || (n[k] > 0 && (n[keep] == 0 || mean[k] > mean[keep]))))
                keep = k;
        if (keep >= 0) act1[keep] = 1;
    }
}

static void apply_pending(ora_t *o, int i, const double *r)
{
    int a = o->aprev[i];
    if (a < 0) return;
    if (r == NULL || !isfinite(r[i])) { o->bad[i] += 1; return; }
    update_arm(o, i, a, o->xprev + (size_t)i * o->d, r[i]);
    if (o->exploit && o->mode[i] < 0) page_hinkley(o, i, o->t, r[i]);
}

double ora_alpha(const void *h, long t)
{
    const ora_t *o = (const ora_t *)h;
    return o->sched == 0 ? o->alpha0 : o->alpha0 / sqrt((double)t + 1.0);
}

/*
 * One decision for every instance.
 *   x      [B][d] context x_t
 *   r      [B]    reward of the previous decision (may be NULL when none is pending)
 *   ucb, lcb [B][K] out: scores of the arms of the action space after rules
 *                   2-8 (before rule 1), -INFINITY for the others
 *   keep   [B][K] out: arms no pruning rule has removed, after this step's
 *                   pruning (the refinement window is not applied to it)
 *   action [B]    out: a_t, or -1 when x_t is not finite
 * The state's action set and last decision are not changed here: see ora_commit.
 */
void ora_decide(void *h, const double *x, const double *r, double *ucb, double *lcb,
                unsigned char *keep, int *action)
{
    ora_decide_ex(h, x, r, ucb, lcb, keep, action, NULL);
}

/* ora_decide, also returning the rule-2/4 margins [B][K] (may be NULL). */
void ora_decide_ex(void *h, const double *x, const double *r, double *ucb, double *lcb,
                   unsigned char *keep, int *action, double *margins)
{
    ora_t *o = (ora_t *)h;
    const int B = o->B, K = o->K, d = o->d;
    const long t = o->t;
    const int pending = o->pending;
    const double alpha = ora_alpha(o, t);
    const int prune_now = (o->prune & 1) && t > 0 && (t % o->period) == 0;
#pragma omp parallel for schedule(dynamic, 4)
    for (int i = 0; i < B; ++i) {
        if (pending) apply_pending(o, i, r);
        const double *xi = x + (size_t)i * d;
        unsigned char act0[1024], act1[1024];
        double marg[1024];
        const unsigned char *glob = o->active + (size_t)i * K;
        double *U = ucb + (size_t)i * K, *L = lcb + (size_t)i * K;
        unsigned char *kp = keep + (size_t)i * K;
        for (int k = 0; k < K; ++k) {
            U[k] = -INFINITY; L[k] = -INFINITY; kp[k] = glob[k]; marg[k] = INFINITY;
            act0[k] = glob[k] && in_space(o, i, k);
        }
        const unsigned char *act = act0;   /* the action space: not pruned, in the window */
        if (!all_finite(xi, d)) {
            o->bad[i] += 1;
            action[i] = -1;
            if (margins) memcpy(margins + (size_t)i * K, marg, sizeof(double) * K);
            continue;
        }
        if (o->exploit && o->mode[i] < 0 && t >= o->ph_min_rounds && t - o->ph_last[i] >= o->ph_window)
            o->mode[i] = t;
        const int greedy = o->mode[i] >= 0;
        if (prune_now && !o->sticky && !greedy)
            for (int k = 0; k < K; ++k) {   /* rule 1 starts again from the whole space */
                kp[k] = 1;
                act0[k] = in_space(o, i, k);
            }
        if (o->prune & 14) {
            heuristic_prune(o, i, t, act, act1, marg);
            for (int k = 0; k < K; ++k)
                if (act0[k] && !act1[k]) kp[k] = 0;
            act = act1;
        }
        if (margins) memcpy(margins + (size_t)i * K, marg, sizeof(double) * K);
        for (int k = 0; k < K; ++k) {
            if (!act[k]) continue;
            size_t ik = (size_t)i * K + k;
            const double *Ainv = o->Ainv + ik * d * d, *theta = o->theta + ik * d;
            double m = 0.0, quad = 0.0;
            for (int p = 0; p < d; ++p) m += theta[p] * xi[p];
            for (int p = 0; p < d; ++p) {
                double row = 0.0;
                for (int q = 0; q < d; ++q) row += Ainv[p * d + q] * xi[q];
                quad += xi[p] * row;
            }
            double w = sqrt(quad > 0.0 ? quad : 0.0);
            U[k] = greedy ? m : m + alpha * w;   /* Eq. 2 when exploiting, else Eq. 1 */
            L[k] = greedy ? m : m - alpha * w;
        }
        if (prune_now && !greedy) {
            double lstar = -INFINITY;
            for (int k = 0; k < K; ++k)
                if (act[k] && L[k] > lstar) lstar = L[k];
            for (int k = 0; k < K; ++k)
                if (act[k] && U[k] < lstar) kp[k] = 0;
        }
        int best = -1;
        for (int k = 0; k < K; ++k)
            if (act[k] && kp[k] && (best < 0 || U[k] > U[best])) best = k;
        action[i] = best;
    }
    o->pending = 0;
}

/* Refinement of instance i's action space after the decision a of step t. */
static void refine_space(ora_t *o, int i, long t, int a)
{
    const int K = o->K;
    const unsigned char *glob = o->active + (size_t)i * K;
    const int *n = o->nsel + (size_t)i * K;
    const double *rs = o->rsum + (size_t)i * K;
    int anchor = -1;
    if (t < o->refine_mature) {
        /* statistical: best mean reward (lowest mean EDP), enough samples */
        for (int k = 0; k < K; ++k)
            if (glob[k] && in_space(o, i, k) && n[k] >= o->refine_min_n &&
                (anchor < 0 || rs[k] / n[k] > rs[anchor] / n[anchor]))
                anchor = k;
    } else {
        anchor = a;   /* predictive: this step's UCB (or Eq. 2) argmax */
    }
    if (anchor < 0) return;
    o->win[3 * i] = anchor - o->refine_half > 0 ? anchor - o->refine_half : 0;
    o->win[3 * i + 1] = anchor + o->refine_half < K - 1 ? anchor + o->refine_half : K - 1;
    o->win[3 * i + 2] = 1;
}

/* Record the decision taken at this step: x_t, a_t and the arms no pruning
 * rule has removed; then refine the action space when due. */
void ora_commit(void *h, const double *x, const int *action, const unsigned char *keep)
{
    ora_t *o = (ora_t *)h;
    const int B = o->B, K = o->K, d = o->d;
    const long t = o->t;
    const int refine_now = o->refine && t > 0 && (t % o->refine_period) == 0;
    for (int i = 0; i < B; ++i) {
        memcpy(o->xprev + (size_t)i * d, x + (size_t)i * d, sizeof(double) * d);
        o->aprev[i] = action[i];
        if (keep) memcpy(o->active + (size_t)i * K, keep + (size_t)i * K, K);
        if (refine_now && action[i] >= 0) refine_space(o, i, t, action[i]);
    }
    o->t += 1;
    o->pending = 1;
}

/* Apply the last pending update (rewards of the final decisions). */
void ora_flush(void *h, const double *r)
{
    ora_t *o = (ora_t *)h;
    if (o->pending)
        for (int i = 0; i < o->B; ++i) apply_pending(o, i, r);
    o->pending = 0;
    for (int i = 0; i < o->B; ++i) o->aprev[i] = -1;
}

/* Copy out instance i's state; any output pointer may be NULL. */
void ora_get(const void *h, int i, double *A, double *b, double *Ainv, double *theta,
             unsigned char *active, int *nsel, int *bad)
{
    ora_get_rsum(h, i, NULL);
    const ora_t *o = (const ora_t *)h;
    const int K = o->K, d = o->d;
    size_t base = (size_t)i * K;
    if (A) memcpy(A, o->A + base * d * d, sizeof(double) * K * d * d);
    if (b) memcpy(b, o->b + base * d, sizeof(double) * K * d);
    if (Ainv) memcpy(Ainv, o->Ainv + base * d * d, sizeof(double) * K * d * d);
    if (theta) memcpy(theta, o->theta + base * d, sizeof(double) * K * d);
    if (active) memcpy(active, o->active + base, K);
    if (nsel) memcpy(nsel, o->nsel + base, sizeof(int) * K);
    if (bad) *bad = o->bad[i];
}

/* Sum of the rewards folded into each arm of instance i ([K]). */
void ora_get_rsum(const void *h, int i, double *rsum)
{
    const ora_t *o = (const ora_t *)h;
    if (rsum) memcpy(rsum, o->rsum + (size_t)i * o->K, sizeof(double) * o->K);
}

long ora_t_now(const void *h) { return ((const ora_t *)h)->t; }

int ora_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void ora_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
